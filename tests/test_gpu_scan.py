"""GPU parity of the one-pass MFMA scoring kernel (16 or more queries per head
over at least 16,384 keys: batches of decode queries over a long cache)
against the float64 oracle, through the C ABI."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from tests.test_gpu_parity import _t, check_head, gpu_pipeline, oracle_factors

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2608_03228_amd.saki")

pytestmark = pytest.mark.gpu

MODE = {"f32": "f32", "bf16": "bf16_emul", "fp8": "fp8_emul"}


@pytest.mark.parametrize("sketch,r,Q,N,batch", [
    ("bf16", 32, 16, 40_003, 1),   # key axis in chunks, ragged last tile
    ("f32", 16, 20, 17_000, 2),    # two sequences, a second row block of 4 rows
    ("fp8", 64, 33, 20_000, 1),    # three row blocks, the last with one row
    ("bf16", 128, 16, 16_384, 1),  # the shortest rows that take this kernel
])
def test_scan_matches_oracle(sketch, r, Q, N, batch):
    """Fresh queries over all keys; every row of every head checked."""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=N, Q=Q, H_q=2, H_kv=1, batch=batch)
    inp = W.make_layer(spec)
    out = gpu_pipeline(inp, r, sketch)
    for b in range(batch):
        for h in range(2):
            n, ex, diff = check_head(inp, out, b, h, r, MODE[sketch])
            print(f"b{b} h{h}: rows {n} exempt {ex} differing {diff}")
            assert diff == 0


def test_scan_positions_n_valid_and_small_k():
    """Rows limited to their own positions (from 100 keys to all of them),
    N_valid below N_cap and k = 10: rows end inside chunks, some chunks hold
    too few of a row's keys for a gate, later chunks none."""
    N_cap, N_valid, Q = 20_000, 19_000, 48
    spec = W.SPECS["qwen25_7b_decode"].with_(N=N_cap, Q=Q, H_q=2, H_kv=1, batch=1)
    inp = W.make_layer(spec)
    pos = np.linspace(99, N_valid + 500, Q).astype(np.int32)  # the last rows see all N_valid
    inp = dict(inp, q_pos=pos)
    out = gpu_pipeline(inp, 32, "bf16", k=10, N_valid=N_valid, q_pos=pos)
    for h in range(2):
        check_head(inp, out, 0, h, 32, "bf16_emul", k=10, N_valid=N_valid)


def _planted(inp, plants):
    """Replace keys: for each (row, positions, scores) triple, the keys at
    those positions become mu + a u with u = M^T q_row (M = B_q B_k^T of head
    0), a chosen so that each scores the given value for that row (on the
    oracle's float64 scores).  Returns the new inputs and head 0's scores."""
    keys = inp["keys"].copy()
    Bq, Bk, mu = oracle_factors(inp, 0, 32)
    M = Bq @ Bk.T
    q = inp["queries"][0, 0].astype(np.float64)
    for i, pos, score in plants:
        u = M.T @ q[i]
        for j, sc in zip(pos, score):
            a = (sc - q[i] @ mu) / (u @ u)
            keys[0, 0, j] = (mu + a * u).astype(np.float32)
    s1, *_ = O.index_scores(Bq, Bk, mu, q, keys[0, 0])
    return dict(inp, keys=keys), s1


def _spiked(inp, rows_spikes):
    """Spikes: keys that score about ten times the largest ordinary score for
    their row, each a little apart; checks on the oracle that each outscores
    every ordinary key for its row."""
    Bq, Bk, mu = oracle_factors(inp, 0, 32)
    s0, *_ = O.index_scores(Bq, Bk, mu, inp["queries"][0, 0], inp["keys"][0, 0])
    big = 10.0 * np.abs(s0).max()
    out, s1 = _planted(inp, [(i, pos, big * (1.0 + 0.01 * np.arange(len(pos))))
                             for i, pos in rows_spikes])
    every = np.concatenate([p for _, p in rows_spikes])
    plain = np.setdiff1d(np.arange(s1.shape[1]), every)
    for i, pos in rows_spikes:
        assert s1[i, pos].min() > s1[i, plain].max()
    return out


def _sampled(chunk0, tile, g, v):
    """Key sampled by lane group g (element v) in the gate's sampled tile
    `tile` of a 2,048-key chunk (sampled every 256 keys)."""
    return chunk0 + 256 * tile + 4 * g + v


def test_scan_short_chunks_pass_the_merged_check():
    """Row 0's sampled keys in the first tile of chunks 0 and 5 are replaced
    by keys that score near its 90th-best score, two per lane group: the gate
    of those chunks sits there, so they keep fewer than 64 keys, while more
    than 64 keys of the row lie above it and the merged list passes the
    check.  (16 rows of one head over 16,384 keys are cut into chunks of
    2,048 keys, sampled every 256 keys; lane group g of a row samples keys
    4g .. 4g + 3 of each 16 of a tile.)"""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=16_384, Q=16, H_q=2, H_kv=1, batch=1)
    inp = W.make_layer(spec)
    Bq, Bk, mu = oracle_factors(inp, 0, 32)
    s0, *_ = O.index_scores(Bq, Bk, mu, inp["queries"][0, 0], inp["keys"][0, 0])
    top = np.sort(s0[0])[::-1]
    pos = np.array([_sampled(2048 * c, 0, g, v) for c in (0, 5) for g in range(4) for v in range(2)])
    inp, s1 = _planted(inp, [(0, pos, np.linspace(top[95], top[85], len(pos)))])
    for c in (0, 5):
        assert np.sum(s1[0, 2048 * c:2048 * (c + 1)] > s1[0, pos].min()) < 64
    assert np.sum(s1[0] > s1[0, pos].max()) >= 64
    for sketch in ("f32", "bf16"):
        out = gpu_pipeline(inp, 32, sketch)
        for h in range(2):
            check_head(inp, out, 0, h, 32, MODE[sketch])


def test_scan_spikes_in_two_chunks_are_rescanned():
    """Rows 0..3 get eight keys each, in the sampled tiles of chunks 0 and 5,
    that score far above every other key: those chunks' gates sit on them, no
    other key lies above, and the rows fail the merged check, so their chunks
    are scanned again without a gate."""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=16_384, Q=16, H_q=2, H_kv=1, batch=1)
    inp = W.make_layer(spec)
    spikes = [(i, np.array([_sampled(2048 * c, i, g, v) for c in (0, 5) for g in range(4)
                            for v in range(2)])) for i in range(4)]
    inp = _spiked(inp, spikes)
    for sketch in ("f32", "bf16"):
        out = gpu_pipeline(inp, 32, sketch)
        for h in range(2):
            check_head(inp, out, 0, h, 32, MODE[sketch])


def test_scan_rows_failing_the_merged_check_are_rescanned():
    """Row 0's 64 best keys are spikes, eight in the sampled tiles of every
    chunk: each chunk keeps only its spikes above its gate, and the merged
    64th score (the lowest spike) does not lie above every chunk's gate, so
    the row is flagged and its chunks are scanned again without a gate."""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=16_384, Q=16, H_q=2, H_kv=1, batch=1)
    inp = W.make_layer(spec)
    pos = np.array([_sampled(2048 * c, c % 8, g, v) for c in range(8) for g in range(4)
                    for v in range(2)])
    inp = _spiked(inp, [(0, pos)])
    for sketch in ("f32", "bf16"):
        out = gpu_pipeline(inp, 32, sketch)
        assert set(out["idx"][0, 0, 0].tolist()) == set(pos.tolist())
        for h in range(2):
            check_head(inp, out, 0, h, 32, MODE[sketch])


def test_scan_one_chunk_redo_in_the_wave():
    """Enough rows (16 heads x 2,048 queries) that each wave scans a whole
    row of 16,384 keys: rows 0..3 of head 0 get eight spikes each in their
    sampled tiles (every 2,048 keys here), so their gate keeps fewer than 64
    keys and the wave scans them again.  Sampled rows of two heads checked."""
    spec = W.SPECS["qwen25_7b_decode"].with_(N=16_384, Q=2048, H_q=16, H_kv=1, batch=1)
    inp = W.make_layer(spec)
    spikes = [(i, np.array([2048 * i + 4 * g + v for g in range(4) for v in range(2)]))
              for i in range(4)]
    inp = _spiked(inp, spikes)
    out = gpu_pipeline(inp, 32, "bf16")
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([np.arange(20), rng.choice(2048, 30, False)]))
    for h in (0, 9):
        check_head(inp, out, 0, h, 32, "bf16_emul", rows=rows)
