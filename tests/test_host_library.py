"""CPU tests of libsaki: exported symbols, the host float64 calibration
against the oracle, size helpers and argument validation (no GPU calls)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle as O
import workloads as W

S = pytest.importorskip("paper_2608_03228_amd.saki")
HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "saki.h")


@pytest.fixture(scope="module")
def lib():
    return S.lib()


def test_exports_every_declared_symbol(lib):
    text = open(HEADER).read()
    names = sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(saki_\w+)\(", text, re.M)))
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert S.saki_version() == 2
    assert "workspace" in S.saki_status_string(-3)


@pytest.mark.parametrize("n", [1, 2, 3, 17, 128])
def test_sym_eig_matches_lapack(n):
    rng = np.random.default_rng(n)
    A = rng.standard_normal((n, n))
    A = A + A.T
    w, V = S.saki_sym_eig(A)
    w2 = np.linalg.eigvalsh(A)
    scale = np.abs(w2).max()
    assert np.max(np.abs(w - w2)) <= 1e-13 * n * scale
    assert np.max(np.abs(A @ V - V * w)) <= 1e-13 * n * scale
    np.testing.assert_allclose(V.T @ V, np.eye(n), atol=1e-13 * n)


def test_sym_eig_degenerate_and_graded():
    # repeated eigenvalues, exact zeros, and a wide dynamic range
    Q, _ = np.linalg.qr(np.random.default_rng(0).standard_normal((40, 40)))
    w0 = np.concatenate([np.full(10, 2.0), np.zeros(10), np.geomspace(1e-12, 1e3, 20)])
    A = (Q * w0) @ Q.T
    w, V = S.saki_sym_eig(A)
    np.testing.assert_allclose(w, np.sort(w0), atol=1e-12 * 1e3)
    assert np.max(np.abs(A @ V - V * w)) <= 1e-11 * 1e3
    w, V = S.saki_sym_eig(np.diag([3.0, 1.0, 2.0]))
    np.testing.assert_array_equal(w, [1.0, 2.0, 3.0])


@pytest.mark.parametrize("n", [4, 9, 33, 128])
def test_sym_eig_structured_matrices(n):
    """Matrices whose Householder reduction meets columns that are already
    reduced part-way (a zero or diagonal matrix, a block-diagonal one, a
    low-rank one): eigenvalues, residuals and orthogonality as for dense ones."""
    rng = np.random.default_rng(100 + n)
    A = rng.standard_normal((n, n))
    A = A + A.T
    blocks = A.copy()
    blocks[n // 2:, :n // 2] = 0.0
    blocks[:n // 2, n // 2:] = 0.0
    B = rng.standard_normal((n, 2))
    for M in (np.zeros((n, n)), np.diag(rng.standard_normal(n)), blocks, B @ B.T):
        w, V = S.saki_sym_eig(M)
        ref = np.linalg.eigvalsh(M)
        scale = max(np.abs(ref).max(), 1.0)
        assert np.max(np.abs(w - ref)) <= 1e-13 * n * scale
        assert np.max(np.abs(M @ V - V * w)) <= 1e-13 * n * scale
        np.testing.assert_allclose(V.T @ V, np.eye(n), atol=1e-13 * n)


def test_sym_eig_close_pairs_and_split_tridiagonals():
    """Wilkinson's W21+ (its largest eigenvalues come in pairs that agree to
    about 1e-14) and a tridiagonal whose couplings are partly below the
    deflation threshold: eigenvalues against LAPACK, residuals, orthogonality."""
    n = 21
    W = np.diag(np.abs(np.arange(n) - 10.0)) + np.diag(np.ones(n - 1), 1) + np.diag(np.ones(n - 1), -1)
    T = np.diag(np.linspace(-3.0, 5.0, 30)) + np.diag(np.where(np.arange(29) % 3 == 0, 1e-300, 0.5), 1)
    T = np.triu(T) + np.triu(T, 1).T
    for M in (W, T):
        w, V = S.saki_sym_eig(M)
        ref = np.linalg.eigvalsh(M)
        scale = np.abs(ref).max()
        assert np.max(np.abs(w - ref)) <= 1e-13 * len(M) * scale
        assert np.max(np.abs(M @ V - V * w)) <= 1e-13 * len(M) * scale
        np.testing.assert_allclose(V.T @ V, np.eye(len(M)), atol=1e-13 * len(M))


def _m(B_q, B_k):
    return B_q.astype(np.float64) @ B_k.astype(np.float64).T


@pytest.mark.parametrize("spec_name,r", [("single_head_d128", 32), ("llama31_8b_layer", 16),
                                         ("llama31_8b_layer", 64), ("qwen25_7b_decode", 32)])
def test_calibration_matches_oracle(spec_name, r):
    """Host calibration vs the oracle.  The library returns float32 factors, so
    the rank-r map agrees to float32 rounding (~1e-7 relative); singular
    values are float64 throughout (SVD via the eigenvalues of C^T C)."""
    spec = W.SPECS[spec_name].with_(N=64, Q=1, q_start=0, batch=1)
    inp = W.make_layer(spec)
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r)
    G = spec.H_q // spec.H_kv
    for h in sorted({0, spec.H_q // 2, spec.H_q - 1}):
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][h // G], r)
        M = _m(cal["B_q"][h], cal["B_k"][h])
        assert np.linalg.norm(M - oc["M"]) <= 2e-6 * np.linalg.norm(oc["M"])
        sig = oc["sigma"]
        assert np.max(np.abs(cal["sigma"][h] ** 2 - sig ** 2)) <= 1e-12 * sig[0] ** 2 * spec.d
        assert tuple(cal["n_clamped"][h]) == oc["n_clamped"]
        np.testing.assert_allclose(cal["mu"][h // G], oc["mu"], rtol=0,
                                   atol=1e-6 * np.abs(oc["mu"]).max())
        for name in ("B_q", "B_k"):  # columns agree, signs canonicalised alike
            a, b = cal[name][h].astype(np.float64), oc[name]
            assert np.max(np.abs(a - b) / np.abs(b).max(axis=0)) < 1e-5


@pytest.mark.parametrize("spec_name", ["llama31_8b_layer", "qwen25_7b_decode"])
def test_calibration_without_sigma_matches(spec_name):
    """Without the singular-value output the library takes only the r largest
    eigenvalues (bisection instead of QL): the factors agree with the full path
    to float32 rounding, and the top-r singular values with the oracle."""
    spec = W.SPECS[spec_name].with_(N=64, Q=1, q_start=0, batch=1)
    inp = W.make_layer(spec)
    full = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32)
    fast = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, with_sigma=False)
    assert fast["sigma"] is None
    for name in ("B_q", "B_k"):
        a, b = fast[name].astype(np.float64), full[name].astype(np.float64)
        assert np.max(np.abs(a - b) / np.abs(b).max(axis=1, keepdims=True)) < 2e-6
    np.testing.assert_array_equal(fast["mu"], full["mu"])
    np.testing.assert_array_equal(fast["n_clamped"], full["n_clamped"])


def test_calibration_clamps_like_oracle():
    """T < d: both moments are singular and the floor binds."""
    rng = np.random.default_rng(9)
    q = rng.standard_normal((2, 40, 128)).astype(np.float32)
    k = (rng.standard_normal((1, 40, 128)) + 0.25).astype(np.float32)
    cal = S.saki_calibrate(q, k, 128)
    for h in range(2):
        oc = O.saki_calibrate(q[h], k[0], 128)
        assert tuple(cal["n_clamped"][h]) == oc["n_clamped"]
        assert oc["n_clamped"][0] >= 88
        np.testing.assert_allclose(_m(cal["B_q"][h], cal["B_k"][h]), np.eye(128), atol=2e-4)


def test_key_pca_and_weight_svd_factors_match_oracle():
    spec = W.SPECS["llama31_8b_layer"].with_(N=64, Q=1, q_start=0)
    inp = W.make_layer(spec)
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, method="key_pca")
    Bq, Bk = S.saki_weight_svd_factors(inp["W_K"], spec.H_q, 32)
    for h in (0, 13, 31):
        g = h // 4
        _, sk, _ = O.second_moments(inp["q_cal"][h], inp["k_cal"][g])
        V = O.key_pca_factors(sk, 32)
        np.testing.assert_allclose(_m(cal["B_q"][h], cal["B_k"][h]), V @ V.T, atol=2e-6)
        U = O.weight_svd_factors(inp["W_K"][g], 32)
        np.testing.assert_allclose(_m(Bq[h], Bk[h]), U @ U.T, atol=2e-6)


def test_calibration_with_repeated_singular_values():
    """Sigma_q = I and Sigma_k with repeated eigenvalues: the top-r eigenspace
    is unique when the cut falls between distinct values, so M_r (the
    oblique projector onto it) must match even though the individual
    columns are not unique.  Exercises the re-orthogonalisation of close
    eigenvalues in the host eigensolver."""
    rng = np.random.default_rng(3)
    T, d, r = 256, 16, 5
    ones = np.ones((T, 1)) / np.sqrt(T)
    Z = rng.standard_normal((T, 2 * d))
    Z -= ones @ (ones.T @ Z)                        # zero-mean columns
    U, _ = np.linalg.qr(Z)
    Uq, Uk = U[:, :d], U[:, d:]                     # orthonormal, mutually orthogonal
    q = np.sqrt(T) * Uq                             # Sigma_q = I
    s2 = np.array([5, 5, 5, 3, 3, 2, 1, 1, 1, 0.5, 0.5, 0.25, 0.2, 0.2, 0.1, 0.05])
    V, _ = np.linalg.qr(rng.standard_normal((d, d)))
    k = np.sqrt(T) * (Uk * np.sqrt(s2)) @ V.T + 0.3  # centred moment V diag(s2) V^T
    cal = S.saki_calibrate(q[None].astype(np.float32), k[None].astype(np.float32), r)
    oc = O.saki_calibrate(q.astype(np.float32), k.astype(np.float32), r)
    M = _m(cal["B_q"][0], cal["B_k"][0])
    assert np.linalg.norm(M - oc["M"]) <= 1e-5 * np.linalg.norm(oc["M"])
    assert np.linalg.norm(M @ M - M) <= 1e-5 * np.linalg.norm(M)
    np.testing.assert_allclose(cal["sigma"][0] ** 2, oc["sigma"] ** 2, rtol=0, atol=1e-6 * 5)


def test_shared_calibration_matches_oracle():
    """SAKI_METHOD_SHARED: one map per KV group from the pooled query moment,
    copied to every head of the group, equal to the oracle's shared map."""
    spec = W.SPECS["llama31_8b_layer"].with_(N=64, Q=1, q_start=0)
    inp = W.make_layer(spec)
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, method="shared")
    for g in (0, 5):
        oc = O.saki_calibrate_shared(inp["q_cal"][4 * g:4 * g + 4], inp["k_cal"][g], 32)
        for h in range(4 * g, 4 * g + 4):
            M = _m(cal["B_q"][h], cal["B_k"][h])
            assert np.linalg.norm(M - oc["M"]) <= 2e-6 * np.linalg.norm(oc["M"])
            np.testing.assert_array_equal(cal["B_k"][h], cal["B_k"][4 * g])
        sig = oc["sigma"]
        assert np.max(np.abs(cal["sigma"][4 * g] ** 2 - sig ** 2)) <= 1e-12 * sig[0] ** 2 * spec.d
    assert S.saki_score_topk_workspace_bytes(1, 32, 4032, 4096, 32, 64, "bf16", 8) > 0
    assert S.saki_score_topk_workspace_bytes(1, 32, 4032, 4096, 32, 64, "bf16", 5) == 0


@pytest.mark.parametrize("method", ["opt", "shared", "key_pca", "sap_map", "sap_svd"])
def test_calibrate_from_moments_equals_calibrate(method):
    """saki_calibrate_from_moments on the oracle's float64 moments gives the
    factors of saki_calibrate on the tokens (same arithmetic after the
    moments; only their summation order differs)."""
    spec = W.SPECS["llama31_8b_layer"].with_(N=64, Q=1, q_start=0)
    inp = W.make_layer(spec)
    G = spec.H_q // spec.H_kv
    sq = np.stack([O.second_moments(inp["q_cal"][h], inp["k_cal"][h // G])[0]
                   for h in range(spec.H_q)])
    mom = [O.second_moments(inp["q_cal"][0], inp["k_cal"][g]) for g in range(spec.H_kv)]
    sk = np.stack([m[1] for m in mom])
    mu = np.stack([m[2] for m in mom])
    a = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, method=method)
    b = S.saki_calibrate_from_moments(sq, sk, mu, 32, method=method)
    for name in ("B_q", "B_k"):
        x, y = a[name].astype(np.float64), b[name].astype(np.float64)
        assert np.max(np.abs(x - y) / np.abs(y).max(axis=1, keepdims=True)) < 1e-5
    np.testing.assert_allclose(a["mu"], b["mu"], rtol=1e-6, atol=1e-7)
    np.testing.assert_array_equal(a["n_clamped"], b["n_clamped"])


def test_calibration_from_concurrent_callers():
    """Host threads calling the calibration at once share one worker pool:
    jobs are serialised and each caller gets its own, identical, result."""
    import threading
    spec = W.SPECS["llama31_8b_layer"].with_(N=64, Q=1, q_start=0)
    inp = W.make_layer(spec)
    ref = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, n_threads=4)
    out = [None] * 6

    def work(i):
        out[i] = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, n_threads=1 + i % 4)

    ts = [threading.Thread(target=work, args=(i,)) for i in range(len(out))]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    for o in out:
        for name in ("B_q", "B_k", "mu"):
            np.testing.assert_array_equal(o[name], ref[name])


def _calibrate_in_child(conn):
    rng = np.random.default_rng(4)
    q = rng.standard_normal((4, 96, 16)).astype(np.float32)
    k = rng.standard_normal((2, 96, 16)).astype(np.float32)
    conn.send(S.saki_calibrate(q, k, 4, n_threads=3)["B_k"])
    conn.close()


def test_calibration_after_fork():
    """A child forked after the parent started its workers builds its own."""
    import multiprocessing as mp
    rng = np.random.default_rng(4)
    q = rng.standard_normal((4, 96, 16)).astype(np.float32)
    k = rng.standard_normal((2, 96, 16)).astype(np.float32)
    ref = S.saki_calibrate(q, k, 4, n_threads=3)["B_k"]  # parent's workers exist now
    ctx = mp.get_context("fork")
    a, b = ctx.Pipe(duplex=False)
    p = ctx.Process(target=_calibrate_in_child, args=(b,))
    p.start()
    assert a.poll(60), "child calibration did not finish"
    got = a.recv()
    p.join(30)
    assert p.exitcode == 0
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("kind", ["map", "svd"])
def test_sap_factors_match_oracle(kind):
    """SAP-map / SAP-svd bases (Sec. 6) of every head against the oracle's,
    and the projector they define."""
    spec = W.SPECS["llama31_8b_layer"].with_(N=64, Q=1, q_start=0)
    inp = W.make_layer(spec)
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, method="sap_" + kind)
    G = spec.H_q // spec.H_kv
    for h in range(spec.H_q):
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][h // G], 32)
        Q = O.sap_factors(oc, 32, kind)
        np.testing.assert_array_equal(cal["B_q"][h], cal["B_k"][h])
        Bk = cal["B_k"][h].astype(np.float64)
        assert np.max(np.abs(Bk - Q)) < 1e-6
        sig = oc["sigma"]
        assert np.max(np.abs(cal["sigma"][h] ** 2 - sig ** 2)) <= 1e-12 * sig[0] ** 2 * spec.d
    np.testing.assert_allclose(cal["mu"], inp["k_cal"].astype(np.float64).mean(1), rtol=1e-6,
                               atol=1e-7)


def test_constant_keys_identity_fallback():
    q = np.random.default_rng(1).standard_normal((1, 64, 16)).astype(np.float32)
    k = np.tile(np.arange(16, dtype=np.float32), (1, 64, 1))
    cal = S.saki_calibrate(q, k, 4)
    assert cal["n_clamped"][0, 1] == 16
    np.testing.assert_array_equal(cal["mu"][0], np.arange(16, dtype=np.float32))


def test_size_helpers():
    assert S.saki_index_bytes(1, 32, 4096, 32, "bf16") == 32 * 4096 * 32 * 2
    assert S.saki_index_bytes(2, 4, 65, 16, "f32") == 2 * 4 * 128 * 16 * 4  # tiles of 64 keys
    assert S.saki_index_bytes(1, 1, 64, 48, "f32") == 0  # unsupported rank
    assert S.saki_score_topk_workspace_bytes(1, 32, 4032, 4096, 32, 64, "bf16") > 0
    assert S.saki_score_topk_workspace_bytes(1, 32, 4032, 4096, 32, 65, "bf16") == 0
    # decode rows are split over many key chunks -> room for partial lists
    assert S.saki_score_topk_workspace_bytes(1, 32, 1, 1 << 20, 32, 64, "bf16") > 32 * 64 * 8
    assert S.saki_recall_workspace_bytes(1, 32, 8, 1, 1 << 20, 128, 64) > 0
    assert S.saki_recall_workspace_bytes(1, 32, 8, 1, 1 << 20, 64, 64) == 0


def test_scan_workspace_holds_lists_gates_and_flags():
    """16 or more queries per head over at least 16,384 keys take the one-pass
    MFMA scan: with the key axis in chunks its workspace holds, per row, a
    64-entry partial list (8 B each) and a gate (4 B) per chunk, and a redo
    flag (4 B).  The chunk count is the planner's (one per 2,048 waves' worth
    of rows, chunks of at least 2,048 keys), so the bound below follows from
    the sizes alone."""
    B, H, Q, N = 8, 28, 16, 131_072
    rows = B * H * Q
    waves = B * H * (Q // 16)                   # one 16-row block per head
    want = -(-2048 // waves)                    # chunks per row for 2,048 waves
    chunk = max(2048, -(-(-(-N // want)) // 64) * 64)
    chunks = -(-N // chunk)
    assert chunks == 10
    ws = S.saki_score_topk_workspace_bytes(B, H, Q, N, 32, 64, "bf16")
    assert ws >= rows * chunks * (64 * 8 + 4) + rows * 4
    # one row block of one head over 16,384 keys: 8 chunks of 2,048 keys
    ws1 = S.saki_score_topk_workspace_bytes(1, 1, 16, 16_384, 32, 64, "bf16")
    assert ws1 >= 16 * 8 * (64 * 8 + 4) + 16 * 4
    # enough rows that every row block scans its keys in one chunk: no partial
    # lists, gates or flags (the minimum workspace)
    assert S.saki_score_topk_workspace_bytes(1, 16, 2048, 16_384, 32, 64, "bf16") == 256
    # rows shorter than 16,384 keys, 16 or more queries: the query sketches of
    # every row (r bf16 values, r floats for float32 codes, and b) come first
    rows = 32 * 4032
    for sk, zb in (("bf16", 2), ("fp8", 2), ("f32", 4)):
        ws = S.saki_score_topk_workspace_bytes(1, 32, 4032, 4096, 32, 64, sk)
        assert rows * (32 * zb + 4) <= ws <= rows * (32 * zb + 4) + 512
    # and past one 4,096-key chunk the partial lists besides
    ws = S.saki_score_topk_workspace_bytes(2, 8, 64, 10_000, 64, 64, "bf16")
    assert ws >= 2 * 8 * 64 * (3 * 64 * 8 + 64 * 2 + 4)


def test_argument_validation_without_launch(lib):
    """Invalid arguments are rejected before anything touches the GPU."""
    P = C.c_void_p(1)  # never dereferenced: validation fails first
    ERR_ARG, ERR_UNSUP, ERR_WS = -1, -2, -3
    # build_index: d != 128, bad rank, null pointers, range past N_cap, small buffer
    assert lib.saki_build_index(P, 0, 1, 1, 1, 64, 64, 32, P, P, 0, P, 1 << 20, 0, 64, None) == ERR_UNSUP
    assert lib.saki_build_index(P, 0, 1, 1, 1, 64, 128, 48, P, P, 0, P, 1 << 20, 0, 64, None) == ERR_UNSUP
    assert lib.saki_build_index(None, 0, 1, 1, 1, 64, 128, 32, P, P, 0, P, 1 << 20, 0, 64, None) == ERR_ARG
    assert lib.saki_build_index(P, 0, 1, 1, 1, 64, 128, 32, P, P, 0, P, 1 << 20, 10, 60, None) == ERR_ARG
    assert lib.saki_build_index(P, 0, 1, 1, 1, 64, 128, 32, P, P, 0, P, 100, 0, 64, None) == ERR_WS
    assert lib.saki_build_index(P, 0, 1, 3, 2, 64, 128, 32, P, P, 0, P, 1 << 20, 0, 64, None) == ERR_ARG
    assert lib.saki_build_index(P, 7, 1, 1, 1, 64, 128, 32, P, P, 0, P, 1 << 20, 0, 64, None) == ERR_UNSUP
    # score_topk: k out of range, N_valid > N_cap, small workspace, null output
    args = [P, 0, 1, 1, 1, 1, 256, 256, 128, 32, P, None, 4, P, P]
    assert lib.saki_score_topk(*args, 65, P, None, P, 1 << 30, None) == ERR_UNSUP
    assert lib.saki_score_topk(*args, 0, P, None, P, 1 << 30, None) == ERR_UNSUP
    assert lib.saki_score_topk(*args, 64, None, None, P, 1 << 30, None) == ERR_ARG
    assert lib.saki_score_topk(*args, 64, P, None, P, 1, None) == ERR_WS
    bad = [P, 0, 1, 1, 1, 1, 256, 300, 128, 32, P, None, 4, P, P]
    assert lib.saki_score_topk(*bad, 64, P, None, P, 1 << 30, None) == ERR_ARG
    # Q == 0 is a no-op that succeeds
    zero = [P, 0, 1, 1, 1, 1, 256, 256, 128, 32, P, None, 0, P, P]
    assert lib.saki_score_topk(*zero, 64, P, None, P, 0, None) == 0
    # index heads must divide H_q and be a multiple of H_kv (here H_q = 8, H_kv = 2)
    for ih in (0, 3, 1, 16):
        gqa = [P, 0, 1, 8, 2, ih, 256, 256, 128, 32, P, None, 4, P, P]
        assert lib.saki_score_topk(*gqa, 64, P, None, P, 1 << 30, None) == ERR_ARG, ih
    # the allocation-free variant: same validation; a call needing more than
    # its static scratch array fails before the array is touched
    na = [P, 0, 1, 1, 1, 1, 256, 256, 128, 32, P, None, 4, P, P]
    assert lib.saki_score_topk_noalloc(*na, 65, P, None, None) == ERR_UNSUP
    assert lib.saki_score_topk_noalloc(*na, 64, None, None, None) == ERR_ARG
    # 2,047 heads x 16 queries over 16,384 keys: two key chunks per row, whose
    # partial lists, gates and flags need just over 32 MiB
    need = S.saki_score_topk_workspace_bytes(1, 2047, 16, 16_384, 32, 64, "bf16")
    assert need > S.saki_noalloc_scratch_bytes() == 32 << 20
    over = [P, 1, 1, 2047, 1, 2047, 16_384, 16_384, 128, 32, P, None, 16, P, P]
    assert lib.saki_score_topk_noalloc(*over, 64, P, None, None) == ERR_WS
    # recall: null hits, bad key dtype
    assert lib.saki_recall(P, 0, P, None, 1, 1, 1, 256, 256, 4, 128, 64, P, None, None, P,
                           1 << 30, None) == ERR_ARG
    assert lib.saki_recall(P, 3, P, None, 1, 1, 1, 256, 256, 4, 128, 64, P, P, None, P,
                           1 << 30, None) == ERR_UNSUP
    # attend: k > 64, d != 128, bad key source, no valid key, missing index
    #   (keys, key_dtype, values, index, sketch, source, B, H_q, H_kv, index_heads,
    #    N_cap, N_valid, d, r, q, q_pos, Q, B_q, mu, top_idx, k, theta, out, stream)
    def attend(**kw):
        a = dict(keys=P, key_dtype=0, values=P, index=P, sketch=1, source=0, B=1, H_q=2, H_kv=1,
                 index_heads=2, N_cap=256, N_valid=256, d=128, r=32, q=P, q_pos=None, Q=4, B_q=P,
                 mu=P, top_idx=P, k=64, theta=500000.0, out=P)
        a.update(kw)
        return lib.saki_attend(*a.values(), None)
    assert attend(k=65) == ERR_UNSUP
    assert attend(d=64) == ERR_UNSUP
    assert attend(source=2) == ERR_ARG
    assert attend(N_valid=0) == ERR_ARG
    assert attend(theta=0.0) == ERR_ARG
    assert attend(keys=None) == ERR_ARG
    assert attend(source=1, index=None) == ERR_ARG
    assert attend(source=1, r=48) == ERR_UNSUP
    assert attend(source=1, index_heads=3) == ERR_ARG
    assert attend(key_dtype=2) == ERR_UNSUP  # fp8 is a code type, not a key type
    assert attend(Q=0) == 0
    # calibration: H_q not a multiple of H_kv, r > d, null output
    f = np.zeros((2, 8, 4), np.float32)
    out = np.zeros(64, np.float32)
    fp = f.ctypes.data
    assert lib.saki_calibrate(fp, fp, 3, 2, 8, 4, 2, 0, 1e-6, out.ctypes.data, out.ctypes.data,
                              out.ctypes.data, None, None, 1) == ERR_ARG
    assert lib.saki_calibrate(fp, fp, 2, 2, 8, 4, 5, 0, 1e-6, out.ctypes.data, out.ctypes.data,
                              out.ctypes.data, None, None, 1) == ERR_ARG
    assert lib.saki_calibrate(fp, fp, 2, 2, 8, 4, 2, 0, 1e-6, None, out.ctypes.data,
                              out.ctypes.data, None, None, 1) == ERR_ARG
    assert lib.saki_calibrate(fp, fp, 2, 2, 8, 4, 2, 9, 1e-6, out.ctypes.data, out.ctypes.data,
                              out.ctypes.data, None, None, 1) == ERR_UNSUP


def test_nonfinite_calibration_input_is_reported():
    q = np.ones((1, 16, 8), np.float32)
    q[0, 3, 2] = np.nan
    with pytest.raises(S.SakiError) as e:
        S.saki_calibrate(q, np.ones((1, 16, 8), np.float32), 2)
    assert e.value.status == -6
