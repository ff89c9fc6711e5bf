"""SAKI oracle: calibration, codes, sketch scores, top-k and recall in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Each function states
the passage of the paper it follows.  Notation follows the paper: per head,
Sigma_q is the uncentred second moment of the queries, Sigma_k and mu the
centred second moment and mean of the keys, C = Sigma_q^{1/2} Sigma_k^{1/2}
(Eq. 2), C_r = U_r Lambda_r V_r^T its rank-r truncated SVD, and the optimal
rank-r score map is M_r = Sigma_q^{-1/2} C_r Sigma_k^{-1/2} (Eq. 3,
Proposition 1).  Keys are stored as codes c = B_k^T (k - mu) and a query
scores them as (B_q^T q)^T c + q^T mu (Eq. 4, Sec. 6).

Readings taken where the paper is silent (listed with reasons in the design
notes): moments use the 1/T normaliser; eigenvalues of each Sigma below
floor_rel * lambda_max are clamped to that floor (never truncated); singular
vector pairs are sign-canonicalised so that the largest-magnitude entry of each
column of B_k is positive (lowest index on ties); top-k ranks by score
descending, then key index ascending.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "second_moments", "clamped_roots", "saki_calibrate", "saki_calibrate_shared",
    "key_pca_factors", "sap_factors",
    "weight_svd_factors", "score_loss", "codes", "query_sketch", "sketch_scores",
    "direct_scores", "exact_scores", "candidate_limits", "topk_row", "topk_rows",
    "recall_hits", "bf16_round", "f32_round", "fp8_round", "E4M3_MAX", "score_scale",
    "norm_scale",
    "predicted_reduction", "measured_reduction", "population_reduction",
    "head_group", "index_scores", "PAD_IDX", "ROPE_THETA", "rope", "reconstruct_keys",
    "sparse_attention",
]

PAD_IDX = -1


def head_group(h: int, H_q: int, H_kv: int) -> int:
    """GQA: query head h reads KV head floor(h / (H_q / H_kv)) (Sec. 3)."""
    return h // (H_q // H_kv)


def second_moments(q_cal: np.ndarray, k_cal: np.ndarray):
    """Calibration moments of one head (Sec. 6; Appendix A, centring).

    q_cal [T, d], k_cal [T, d].  Returns (Sigma_q, Sigma_k, mu): Sigma_q is the
    uncentred second moment of the queries, Sigma_k the second moment of the
    centred keys k - mu, mu the key mean; all with the 1/T normaliser.
    """
    q = np.asarray(q_cal, np.float64)
    k = np.asarray(k_cal, np.float64)
    T = q.shape[0]
    sq = q.T @ q / T
    mu = k.sum(axis=0) / T
    kc = k - mu
    sk = kc.T @ kc / T
    return sq, sk, mu


def clamped_roots(S: np.ndarray, floor_rel: float = 1e-6):
    """Symmetric square root and inverse square root of a PSD moment.

    Appendix A (singular covariances, finite-sample regularisation): the
    eigenvalues below floor_rel * lambda_max are raised to that floor, so the
    regularised moment is always invertible.  A moment whose largest
    eigenvalue is not positive (e.g. constant keys) carries no information;
    it is replaced by the identity (every eigenvalue counted as clamped).
    Returns (S^{1/2}, S^{-1/2}, n_clamped).
    """
    S = np.asarray(S, np.float64)
    w, V = np.linalg.eigh(0.5 * (S + S.T))
    lmax = w.max()
    if not lmax > 0.0:
        w = np.ones_like(w)
        n = w.size
    else:
        floor = floor_rel * lmax
        n = int(np.count_nonzero(w < floor))
        w = np.maximum(w, floor)
    half = (V * np.sqrt(w)) @ V.T
    ihalf = (V / np.sqrt(w)) @ V.T
    return half, ihalf, n


def _canonical_signs(U: np.ndarray, V: np.ndarray, Sk_ihalf: np.ndarray):
    """Flip each singular pair (u_i, v_i) so that the largest-|.| entry of the
    key factor column Sigma_k^{-1/2} v_i is positive (first index on ties).
    M_r does not depend on these signs; tying them to B_k rather than to v_i
    makes the stored codes independent of which square root of the moments a
    calibration uses (Eq. 3 is invariant to that choice)."""
    U = U.copy()
    V = V.copy()
    W = Sk_ihalf @ V
    for i in range(V.shape[1]):
        j = int(np.argmax(np.abs(W[:, i])))  # first index on ties
        if W[j, i] < 0:
            U[:, i] = -U[:, i]
            V[:, i] = -V[:, i]
    return U, V


def saki_calibrate(q_cal: np.ndarray, k_cal: np.ndarray, r: int,
                   floor_rel: float = 1e-6) -> dict:
    """SAKI-opt calibration of one query head (Eq. 2-4, Proposition 1, Sec. 6).

    q_cal [T, d] are this head's calibration queries, k_cal [T, d] its KV
    group's calibration keys.  Steps, in the paper's order: moments; clamped
    roots; C = Sigma_q^{1/2} Sigma_k^{1/2}; SVD C = U Lambda V^T;
    B_q = Sigma_q^{-1/2} U_r Lambda_r^{1/2}, B_k = Sigma_k^{-1/2} V_r Lambda_r^{1/2};
    M_r = B_q B_k^T; optimum loss = sum of squared tail singular values.
    """
    sq, sk, mu = second_moments(q_cal, k_cal)
    return _calibrate_from_moments(sq, sk, mu, r, floor_rel)


def saki_calibrate_shared(q_cals: np.ndarray, k_cal: np.ndarray, r: int,
                          floor_rel: float = 1e-6) -> dict:
    """One rank-r map shared by the G query heads of a KV group.

    Extension beyond the paper, which optimises each head on its own: the
    group's summed objective sum_h L_h(P) of Eq. 2 is linear in Sigma_q, so it
    equals G * L(P) for the pooled moment Sigma_q = (1/G) sum_h Sigma_q^(h), and
    Proposition 1 applied to the pooled moment gives the optimal shared map.
    q_cals [G, T, d], k_cal [T, d].
    """
    q_cals = np.asarray(q_cals, np.float64)
    G = q_cals.shape[0]
    sk, mu = second_moments(q_cals[0], k_cal)[1:]
    sq = sum(second_moments(q_cals[h], k_cal)[0] for h in range(G)) / G
    return _calibrate_from_moments(sq, sk, mu, r, floor_rel)


def _calibrate_from_moments(sq, sk, mu, r, floor_rel):
    """The steps of saki_calibrate after the moments."""
    sq_h, sq_ih, nq = clamped_roots(sq, floor_rel)
    sk_h, sk_ih, nk = clamped_roots(sk, floor_rel)
    C = sq_h @ sk_h
    U, sig, Vt = np.linalg.svd(C)
    U, V = _canonical_signs(U, Vt.T, sk_ih)
    root = np.sqrt(sig[:r])
    B_q = sq_ih @ U[:, :r] * root
    B_k = sk_ih @ V[:, :r] * root
    return {
        "Sigma_q": sq, "Sigma_k": sk, "mu": mu,
        "Sq_half": sq_h, "Sq_ihalf": sq_ih, "Sk_half": sk_h, "Sk_ihalf": sk_ih,
        "C": C, "U": U, "sigma": sig, "V": V,
        "B_q": B_q, "B_k": B_k, "M": B_q @ B_k.T,
        "tail": float(np.sum(sig[r:] ** 2)), "n_clamped": (nq, nk),
    }


def key_pca_factors(Sigma_k: np.ndarray, r: int) -> np.ndarray:
    """Key-PCA baseline (Sec. 1, Table 1): the top-r eigenvectors of the
    centred key moment, as the orthonormal basis V [d, r] of the projector
    P = V V^T.  Used with B_q = B_k = V."""
    w, V = np.linalg.eigh(0.5 * (Sigma_k + Sigma_k.T))
    order = np.argsort(-w, kind="stable")
    return V[:, order[:r]]


def _signed_columns(Q: np.ndarray) -> np.ndarray:
    """Flip each column so that its largest-|.| entry is positive (first
    index on ties)."""
    Q = Q.copy()
    for i in range(Q.shape[1]):
        j = int(np.argmax(np.abs(Q[:, i])))
        if Q[j, i] < 0:
            Q[:, i] = -Q[:, i]
    return Q


def sap_factors(cal: dict, r: int, kind: str) -> np.ndarray:
    """Span-projector variants of Sec. 6, as the orthonormal basis Q [d, r] of
    an orthogonal projector P = Q Q^T used with B_q = B_k = Q.

    cal is the output of saki_calibrate (its right singular vectors v_i of
    C = Sigma_q^{1/2} Sigma_k^{1/2} and the root Sigma_k^{1/2}).
    kind "svd" (SAP-svd, the raw right-singular span): span{v_1 .. v_r}.
    kind "map" (SAP-map, the Sigma_k^{1/2}-weighted span, orthonormalised):
    span{Sigma_k^{1/2} v_1 .. Sigma_k^{1/2} v_r}, which is the range of M_r,
    orthonormalised by Gram-Schmidt in the order of the singular values (a
    QR factorisation).  Reading: the paper names both in one line; the basis
    is fixed by signing each column so that its largest-|.| entry is positive,
    and the scores do not depend on the basis, only on P."""
    V = cal["V"][:, :r]
    if kind == "svd":
        Q = V
    elif kind == "map":
        Q, _ = np.linalg.qr(cal["Sk_half"] @ V)
    else:
        raise ValueError(kind)
    return _signed_columns(Q)


def weight_svd_factors(W_K: np.ndarray, r: int) -> np.ndarray:
    """Weight-SVD baseline (Sec. 1, Table 1; reading: data-blind truncation of
    the key projection): top-r left singular vectors U [d, r] of W_K [d, D],
    used as B_q = B_k = U (P = U U^T)."""
    U, _, _ = np.linalg.svd(np.asarray(W_K, np.float64), full_matrices=False)
    return U[:, :r]


def score_loss(P: np.ndarray, Sq_half: np.ndarray, Sk_half: np.ndarray) -> float:
    """Expected squared score error of a key-side map P in head space (Eq. 2):
    || Sigma_q^{1/2} (I - P) Sigma_k^{1/2} ||_F^2."""
    d = P.shape[0]
    E = Sq_half @ (np.eye(d) - P) @ Sk_half
    return float(np.sum(E * E))


def codes(B_k: np.ndarray, mu: np.ndarray, keys: np.ndarray) -> np.ndarray:
    """Key codes c_j = B_k^T (k_j - mu) (Eq. 4).  keys [..., N, d] -> [..., N, r]."""
    kc = np.asarray(keys, np.float64) - np.asarray(mu, np.float64)
    return kc @ np.asarray(B_k, np.float64)


def query_sketch(B_q: np.ndarray, mu: np.ndarray, q: np.ndarray):
    """Query side of Eq. 4: z = B_q^T q and the exact mean term b = q^T mu."""
    q = np.asarray(q, np.float64)
    return q @ np.asarray(B_q, np.float64), q @ np.asarray(mu, np.float64)


def sketch_scores(z: np.ndarray, b: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Approximate scores s_hat_ij = z_i . c_j + b_i (Sec. 6).  [Q, r], [Q], [N, r] -> [Q, N]."""
    return np.asarray(z, np.float64) @ np.asarray(c, np.float64).T + np.asarray(b)[:, None]


def direct_scores(q: np.ndarray, M: np.ndarray, mu: np.ndarray, keys: np.ndarray) -> np.ndarray:
    """The same scores by the direct route q^T M_r (k - mu) + q^T mu (Sec. 6)."""
    q = np.asarray(q, np.float64)
    kc = np.asarray(keys, np.float64) - mu
    return q @ M @ kc.T + (q @ mu)[:, None]


def exact_scores(q: np.ndarray, keys: np.ndarray) -> np.ndarray:
    """Exact attention logits s_ij = q_i^T k_j (Sec. 3), float64."""
    return np.asarray(q, np.float64) @ np.asarray(keys, np.float64).T


def candidate_limits(Q: int, N: int, q_pos=None) -> np.ndarray:
    """Number of visible keys per query row: all N, or the causal prefix
    j <= position (inclusive, 0-based), capped at N."""
    if q_pos is None:
        return np.full(Q, N, np.int64)
    return np.minimum(np.asarray(q_pos, np.int64) + 1, N)


def topk_row(s: np.ndarray, limit: int, k: int = 64) -> np.ndarray:
    """Top-k of one row by (score descending, key index ascending) over keys
    j < limit, by a full stable sort (Sec. 3 protocol; ties to the lower index).
    Rows with fewer than k candidates are padded with PAD_IDX."""
    n = int(limit)
    j = np.arange(n)
    order = np.lexsort((j, -np.asarray(s[:n], np.float64)))
    out = np.full(k, PAD_IDX, np.int64)
    m = min(k, n)
    out[:m] = order[:m]
    return out


def topk_rows(S: np.ndarray, limits: np.ndarray, k: int = 64) -> np.ndarray:
    """topk_row for every row of S [Q, N]."""
    return np.stack([topk_row(S[i], limits[i], k) for i in range(S.shape[0])])


def recall_hits(approx_idx: np.ndarray, exact_idx: np.ndarray) -> np.ndarray:
    """hits_i = |S_i intersect T_i| per row (Sec. 3: recall of the true top-k),
    by Python set intersection; padding entries never count."""
    a = np.asarray(approx_idx)
    e = np.asarray(exact_idx)
    out = np.empty(a.shape[:-1], np.int64)
    for pos in np.ndindex(*a.shape[:-1]):
        sa = {int(x) for x in a[pos] if x != PAD_IDX}
        se = {int(x) for x in e[pos] if x != PAD_IDX}
        out[pos] = len(sa & se)
    return out


# ---------------------------------------------------------------- reading the winners

ROPE_THETA = 500000.0  # RoPE base of the LLaMA-3.1 models of Sec. 7


def rope(x: np.ndarray, pos, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotary position embedding, rotate-half convention: for m < d/2 the pair
    (x_m, x_{m + d/2}) is rotated by the angle pos * theta^(-2m/d).  Sec. 3:
    codes are built from pre-RoPE keys and the rotation is applied after
    reconstruction.  x [..., d], pos broadcast against x[..., 0]."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, np.float64)[..., None] * inv
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def reconstruct_keys(B_q: np.ndarray, mu: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Sec. 6: k_hat = mu + M_r (k - mu) = mu + B_q c from the stored codes c
    (M_r = B_q B_k^T).  c [N, r] -> [N, d]."""
    return np.asarray(mu, np.float64) + np.asarray(c, np.float64) @ np.asarray(B_q, np.float64).T


def sparse_attention(q, q_pos, keys, values, idx, theta: float = ROPE_THETA) -> np.ndarray:
    """Attention of each query over the keys its index selected (Sec. 1: the
    index nominates candidates, exact values are fetched for the winners), in
    RoPE space: s_j = rope(q, p_q) . rope(k_j, j) / sqrt(d) for the selected j
    (idx >= 0; a key's position is its index), p = softmax(s), out = sum_j p_j v_j.
    q [Q, d], q_pos [Q], keys and values [N, d], idx [Q, k] -> [Q, d]."""
    q = np.asarray(q, np.float64)
    d = q.shape[-1]
    out = np.zeros((q.shape[0], d))
    for i in range(q.shape[0]):
        sel = np.asarray(idx[i])
        sel = sel[sel >= 0]
        if sel.size == 0:
            continue
        qr = rope(q[i], q_pos[i], theta)
        kr = rope(np.asarray(keys, np.float64)[sel], sel, theta)
        sc = kr @ qr / np.sqrt(d)
        w = np.exp(sc - sc.max())
        out[i] = (w / w.sum()) @ np.asarray(values, np.float64)[sel]
    return out


def f32_round(x: np.ndarray) -> np.ndarray:
    """Round to the nearest float32 (ties to even), returned as float64."""
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Storage of a sketch in bf16: round to float32, then to the nearest bf16
    (8-bit significand), ties to even; returned as float64.  Non-finite inputs
    are not supported."""
    f = np.ascontiguousarray(np.asarray(x, np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


def _e4m3_magnitudes() -> np.ndarray:
    """The non-negative finite values of the fp8 E4M3 format (OCP: 1 sign, 4
    exponent bits with bias 7, 3 mantissa bits, subnormals, no infinities;
    code 0x7F is NaN), indexed by code 0x00 .. 0x7E, ascending."""
    v = []
    for code in range(0x7F):
        e, m = code >> 3, code & 7
        v.append(m * 2.0 ** -9 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7))
    return np.array(v)


E4M3_MAX = 448.0


def fp8_round(x: np.ndarray) -> np.ndarray:
    """Storage of a code in fp8 E4M3: round to float32, then to the nearest
    finite E4M3 value, ties to the even code; magnitudes above 448 saturate to
    448 (reading: the format has no infinities).  Returned as float64."""
    f = f32_round(x)
    a = np.abs(f)
    vals = _e4m3_magnitudes()
    hi_i = np.clip(np.searchsorted(vals, a, side="left"), 1, vals.size - 1)
    lo_v, hi_v = vals[hi_i - 1], vals[hi_i]
    d_lo, d_hi = a - lo_v, hi_v - a
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi_i % 2 == 0))
    r = np.where(take_hi, hi_v, lo_v)
    r = np.where(a >= E4M3_MAX, E4M3_MAX, r)
    r = np.where(a == 0.0, 0.0, r)
    return np.copysign(r, f)


def score_scale(B_q, B_k, mu, q, keys) -> np.ndarray:
    """Magnitude scale of computing s_hat from (q, k) through the factors:
    S_ij = sum_m (|B_q|^T|q_i|)_m (|B_k|^T|k_j - mu|)_m + |q_i|^T |mu|.
    A forward error analysis of the factored score bounds its rounding error
    by a small multiple of unit roundoff times S_ij; tolerances are stated
    relative to it.  [Q, d], [N, d] -> [Q, N]."""
    aq = np.abs(np.asarray(q, np.float64))
    ak = np.abs(np.asarray(keys, np.float64) - mu)
    zq = aq @ np.abs(B_q)
    ck = ak @ np.abs(B_k)
    return zq @ ck.T + (aq @ np.abs(mu))[:, None]


def norm_scale(B_q, B_k, mu, q, keys) -> np.ndarray:
    """Scale of the sketch-score tolerances: ||z_i||_2 ||c_j||_2 + |b_i| with the
    exact z_i = B_q^T q_i, c_j = B_k^T (k_j - mu) and b_i = q_i^T mu (Sec. 6).
    By Cauchy-Schwarz it bounds |s_hat_ij|, so a relative tolerance on it is a
    relative tolerance on the score's own magnitude.  [Q, d], [N, d] -> [Q, N]."""
    z, b = query_sketch(B_q, mu, q)
    c = codes(B_k, mu, keys)
    return (np.linalg.norm(z, axis=1)[:, None] * np.linalg.norm(c, axis=1)[None, :]
            + np.abs(b)[:, None])


def predicted_reduction(sigma: np.ndarray, r: int) -> float:
    """Predicted relative score-MSE reduction of the rank-r map (Remark 2,
    Appendix C): 1 - sum_{i>r} sigma_i^2 / sum_i sigma_i^2."""
    s2 = np.asarray(sigma, np.float64) ** 2
    return float(1.0 - s2[r:].sum() / s2.sum())


def measured_reduction(q, keys, M, mu, q_pos=None):
    """Measured relative score-MSE reduction of the map M (Appendix C):
    1 - sum (q^T (I - M)(k - mu))^2 / sum (q^T (k - mu))^2 over (query, key)
    pairs, keys centred by the calibration mean, pre-RoPE.  The denominator is
    the error of the rank-0 map, which keeps only the mean term.

    With q_pos None the pairs are (q_i, k_i), one to one (independent pairs
    when the rows are independent draws); the delta-method standard error of
    the ratio is returned with it.  With q_pos, every causal pair j <= q_pos[i]
    counts, and the standard error is None.  q [n, d], keys [n or N, d]."""
    q = np.asarray(q, np.float64)
    kc = np.asarray(keys, np.float64) - np.asarray(mu, np.float64)
    res = kc - kc @ np.asarray(M, np.float64).T  # (I - M)(k - mu), row-wise
    if q_pos is None:
        base = np.einsum("nd,nd->n", q, kc)
        err = np.einsum("nd,nd->n", q, res)
        a, b = np.mean(err ** 2), np.mean(base ** 2)
        se = np.sqrt(np.var(err ** 2 - (a / b) * base ** 2) / q.shape[0]) / b
        return float(1.0 - a / b), float(se)
    mask = np.arange(kc.shape[0])[None, :] <= np.asarray(q_pos)[:, None]
    base = q @ kc.T
    err = q @ res.T
    return float(1.0 - np.sum(err[mask] ** 2) / np.sum(base[mask] ** 2)), None


def population_reduction(M, mu, Sigma_q, Sigma_k) -> float:
    """The reduction measured_reduction converges to on independent pairs
    (Eq. 2 with the population moments): queries with second moment Sigma_q,
    zero-mean keys with covariance Sigma_k, centred by mu, so the keys' second
    moment about mu is Sigma_k + mu mu^T:
    1 - tr((I - M)^T Sigma_q (I - M) K) / tr(Sigma_q K), K = Sigma_k + mu mu^T."""
    d = np.asarray(M).shape[0]
    K = np.asarray(Sigma_k, np.float64) + np.outer(mu, mu)
    E = np.eye(d) - np.asarray(M, np.float64)
    return float(1.0 - np.trace(E.T @ Sigma_q @ E @ K) / np.trace(Sigma_q @ K))


def index_scores(B_q, B_k, mu, q, keys, sketch: str = "f64"):
    """Scores of one head through the stored index (Eq. 4, Sec. 6), with the
    sketch storage emulated: "f64" keeps exact codes; "f32"/"bf16" round the
    codes c and the query sketch z to that storage type; "fp8" rounds the
    codes to fp8 E4M3 and z to bf16 (the mean term b and the sum stay
    float64).  Returns (s_hat [Q, N], z, b, c) after rounding."""
    c = codes(B_k, mu, keys)
    z, b = query_sketch(B_q, mu, q)
    if sketch == "f32":
        c, z = f32_round(c), f32_round(z)
    elif sketch == "bf16":
        c, z = bf16_round(c), bf16_round(z)
    elif sketch == "fp8":  # fp8 E4M3 codes, bf16 query sketch
        c, z = fp8_round(c), bf16_round(z)
    elif sketch != "f64":
        raise ValueError(sketch)
    return sketch_scores(z, b, c), z, b, c
