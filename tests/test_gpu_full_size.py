"""GPU parity at the full sizes of the synthetic workloads, in the launch
configuration a caller uses for them: every row is computed on the GPU and
sampled rows are checked against the float64 oracle.

Candidate lists given to saki_recall for the checked rows come from the
oracle (its bf16-emulated sketch top-64), never from the GPU; the other rows
keep the GPU's own lists, which only feed the GPU kernel."""
import time

import numpy as np
import pytest

import oracle as O
import workloads as W
from tests.test_gpu_parity import _t, check_head, gpu_pipeline, oracle_factors

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2608_03228_amd.saki")

pytestmark = pytest.mark.gpu


def _log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def _check_emul(inp, out, b, h, rows=None):
    """check_head in the bf16-emulating mode with the rigorous swap bound:
    a row whose set differs from the oracle's must be a swap within
    TIGHT_EMUL * T plus the midpoint allowance (asserted by check_rows), and
    each such row is logged with its gap."""
    log = []
    res = check_head(inp, out, b, h, 32, "bf16_emul", rows=rows, tight=True, log=log)
    for i, gap, bnd in log:
        row = i if rows is None else int(np.asarray(rows)[i])
        _log(f"  b{b} h{h} row {row}: swap gap {gap:.3e} within the float32 bound {bnd:.3e}")
    return res


def _oracle_lists(inp, b, h, r, rows, N, factors=None):
    """The oracle's bf16-emulated sketch top-64 and exact top-64 of sampled rows."""
    spec = inp["spec"]
    G = spec.H_q // spec.H_kv
    Bq, Bk, mu = factors if factors is not None else oracle_factors(inp, h, r)
    q = inp["queries"][b, h][rows]
    keys = inp["keys"][b, h // G][:N]
    pos = inp["q_pos"][rows] if inp["q_pos"] is not None else None
    lim = O.candidate_limits(len(rows), N, pos)
    s_hat, *_ = O.index_scores(Bq, Bk, mu, q, keys, "bf16")
    return O.topk_rows(s_hat, lim), O.topk_rows(O.exact_scores(q, keys), lim)


def _check_recall(out, inp, samples, N, r, want_exact_too=True, factors=None):
    """saki_recall over every row; on the sampled (b, h, rows) the oracle's
    sketch lists go in and the hits (and exact top-64) must equal the oracle's."""
    approx = out["idx"].copy()
    want = {}
    for b, h, rows in samples:
        fac = factors(h) if factors is not None else None
        ap, ex = _oracle_lists(inp, b, h, r, rows, N, fac)
        approx[b, h, rows] = ap
        want[(b, h)] = (ex, O.recall_hits(ap, ex))
    approx_t = _t(approx, torch.int32)
    for we in ((False, True) if want_exact_too else (False,)):
        hits, ex_t = S.saki_recall(out["keys"], out["q"], approx_t, N, q_pos=out["pos"],
                                   want_exact=we)
        torch.cuda.synchronize()
        hits = hits.cpu().numpy()
        ex_np = ex_t.cpu().numpy() if we else None
        for b, h, rows in samples:
            ex, wh = want[(b, h)]
            np.testing.assert_array_equal(hits[b, h, rows], wh)
            if we:
                np.testing.assert_array_equal(ex_np[b, h, rows], ex)
        _log(f"recall want_exact={we}: sampled hits equal the oracle's "
             f"(mean {np.mean([want[k][1].mean() for k in want]) / 64:.4f})")


def _check_own_recall(out, inp, samples, N, r, factors=None):
    """saki_recall over the GPU's own sketch lists: on the sampled rows (whose
    sets equal the oracle's, asserted by the caller) the hits, their integer
    total and the recall printed to four decimals equal the oracle's."""
    hits, _ = S.saki_recall(out["keys"], out["q"], _t(out["idx"], torch.int32), N,
                            q_pos=out["pos"], want_exact=False)
    torch.cuda.synchronize()
    hits = hits.cpu().numpy()
    got = want = n_rows = 0
    for b, h, rows in samples:
        fac = factors(h) if factors is not None else None
        ap, ex = _oracle_lists(inp, b, h, r, rows, N, fac)
        wh = O.recall_hits(ap, ex)
        np.testing.assert_array_equal(hits[b, h, rows], wh)
        got += int(hits[b, h, rows].sum())
        want += int(wh.sum())
        n_rows += len(rows)
    assert got == want and f"{got / (64 * n_rows):.4f}" == f"{want / (64 * n_rows):.4f}"
    _log(f"recall of the GPU's own lists on {n_rows} sampled rows: {got} hits, "
         f"{got / (64 * n_rows):.4f} (oracle {want}, {want / (64 * n_rows):.4f})")


def test_full_llama_layer():
    """LLaMA-3.1-8B-shaped layer as the bench runs it: 32 query / 8 KV heads,
    N = 4096, causal rows 64..4095, bf16 codes at r = 32, one build, one
    score and one recall launch for all heads."""
    spec = W.SPECS["llama31_8b_layer"]
    inp = W.make_layer(spec)
    out = gpu_pipeline(inp, 32, "bf16")
    _log("layer scored")
    rng = np.random.default_rng(11)
    rows = np.unique(np.concatenate([[0, 1, 63, 64, 2047, spec.Q - 1],
                                     rng.choice(spec.Q, 200, False)]))
    for h in (0, 13, 31):
        n, ex, diff = _check_emul(inp, out, 0, h, rows=rows)
        _log(f"h{h}: rows {n} exempt {ex} differing {diff}")
        assert ex <= 0.1 * n
    _check_own_recall(out, inp, [(0, h, rows) for h in (0, 13, 31)], spec.N, 32)
    _check_recall(out, inp, [(0, h, rows) for h in (0, 13, 31)], spec.N, 32)


def test_full_decode_1m():
    """Long-context decode: 2^20 cached keys per KV head, 32 query heads with
    one query each, bf16 codes at r = 32 (the key axis split into chunks that
    one launch covers, then merged).  Three heads checked over all keys."""
    spec = W.SPECS["decode_1m"]
    inp = W.make_layer(spec)
    _log("inputs generated")
    out = gpu_pipeline(inp, 32, "bf16")
    _log("decode step scored")
    for h in (0, 13, 31):
        n, ex, diff = _check_emul(inp, out, 0, h)
        _log(f"h{h}: exempt {ex} differing {diff}")
    _check_own_recall(out, inp, [(0, h, np.arange(spec.Q)) for h in (0, 13, 31)], spec.N, 32)
    _check_recall(out, inp, [(0, h, np.arange(spec.Q)) for h in (0, 31)], spec.N, 32)


def test_full_qwen_decode_layer():
    """Qwen2.5-7B-shaped decode layer: 8 sequences, 28 query / 4 KV heads,
    131,072 keys each, 16 fresh queries per (sequence, head) over all keys
    (the MFMA path), bf16 codes at r = 32."""
    spec = W.SPECS["qwen25_7b_decode"]
    inp = W.make_layer(spec)
    _log("inputs generated")
    out = gpu_pipeline(inp, 32, "bf16")
    _log("layer scored")
    samples = [(0, 0), (3, 13), (7, 27)]
    for b, h in samples:
        n, ex, diff = _check_emul(inp, out, b, h)
        _log(f"b{b} h{h}: rows {n} exempt {ex} differing {diff}")
    _check_own_recall(out, inp, [(b, h, np.arange(spec.Q)) for b, h in samples], spec.N, 32)
    _check_recall(out, inp, [(b, h, np.arange(spec.Q)) for b, h in samples[:2]], spec.N, 32,
                  want_exact_too=False)


def test_full_sweep_one_launch():
    """All 32 LLaMA-shaped layers as 1,024 query heads (256 KV heads) in one
    build, one score and one recall launch: N = 4096, causal rows 64..4095,
    bf16 codes at r = 32.  Heads of three layers sampled."""
    spec = W.SPECS["llama31_8b_sweep"]
    layers = [W.make_layer(spec, layer=l) for l in range(spec.layers)]
    _log("inputs generated")
    inp = {
        "spec": spec.with_(H_q=spec.H_q * spec.layers, H_kv=spec.H_kv * spec.layers),
        "q_cal": np.concatenate([x["q_cal"] for x in layers]),
        "k_cal": np.concatenate([x["k_cal"] for x in layers]),
        "keys": np.concatenate([x["keys"] for x in layers], axis=1),
        "queries": np.concatenate([x["queries"] for x in layers], axis=1),
        "q_pos": layers[0]["q_pos"],
    }
    del layers
    assert inp["queries"].shape[1] == 1024 and inp["keys"].shape[1] == 256
    out = gpu_pipeline(inp, 32, "bf16")
    _log("1024 heads scored")
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([[0, 64, spec.Q - 1], rng.choice(spec.Q, 24, False)]))
    heads = (0, 15 * 32 + 13, 31 * 32 + 31)  # layer 0 head 0, layer 15 head 13, layer 31 head 31
    for h in heads:
        n, ex, diff = _check_emul(inp, out, 0, h, rows=rows)
        _log(f"head {h}: rows {n} exempt {ex} differing {diff}")
    _check_own_recall(out, inp, [(0, h, rows) for h in heads], spec.N, 32)
    _check_recall(out, inp, [(0, h, rows) for h in heads], spec.N, 32, want_exact_too=False)


def test_six_chunk_merges_score_and_recall():
    """8 sequences x 48 query heads x 16 queries over 12,000 keys: both the
    MFMA score path and the MFMA recall path cut the key axis into six chunks
    (384 row blocks), so each row's merge runs six waves and its tree has an
    odd level.  Sampled heads checked against the oracle, with the oracle's
    lists given to the recall."""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=12_000, Q=16, H_q=48, H_kv=4, batch=8)
    inp = W.make_layer(spec)
    _log("inputs generated")
    assert S.saki_score_topk_workspace_bytes(8, 48, 16, 12_000, 32, 64, "bf16") >= 8 * 48 * 16 * 6 * 64 * 8
    out = gpu_pipeline(inp, 32, "bf16")
    samples = [(0, 0), (3, 25), (7, 47)]
    for b, h in samples:
        n, ex, diff = _check_emul(inp, out, b, h)
        _log(f"b{b} h{h}: rows {n} exempt {ex} differing {diff}")
    _check_recall(out, inp, [(b, h, np.arange(16)) for b, h in samples], 12_000, 32)
