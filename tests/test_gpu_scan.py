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


def _spiked(inp, rows_spikes):
    """Replace keys by spikes: for each (row, positions) pair, keys at those
    positions become mu + a u with u = M^T q_row (M = B_q B_k^T of head 0), a
    chosen so that they score about ten times the largest ordinary score for
    that row, each a little apart.  Returns the new inputs after checking on
    the oracle that each spike outscores every ordinary key for its row."""
    keys = inp["keys"].copy()
    Bq, Bk, mu = oracle_factors(inp, 0, 32)
    M = Bq @ Bk.T
    q = inp["queries"][0, 0].astype(np.float64)
    s0, *_ = O.index_scores(Bq, Bk, mu, q, keys[0, 0])
    big = 10.0 * np.abs(s0).max()
    for i, pos in rows_spikes:
        u = M.T @ q[i]
        for m, j in enumerate(pos):
            keys[0, 0, j] = (mu + big * (1.0 + 0.01 * m) / np.linalg.norm(u) ** 2 * u).astype(np.float32)
    s1, *_ = O.index_scores(Bq, Bk, mu, q, keys[0, 0])
    every = np.concatenate([p for _, p in rows_spikes])
    plain = np.setdiff1d(np.arange(keys.shape[2]), every)
    for i, pos in rows_spikes:
        assert s1[i, pos].min() > s1[i, plain].max()
    return dict(inp, keys=keys)


def _sampled(chunk0, tile, g, v):
    """Key sampled by lane group g (element v) in the gate's sampled tile
    `tile` of a 2,048-key chunk (sampled every 256 keys)."""
    return chunk0 + 256 * tile + 4 * g + v


def test_scan_chunk_gates_above_their_64th_score():
    """Keys placed so that the sampled tiles of two chunks hold, for rows
    0..3, eight keys that score far above every other key: the gate read off
    the sample then keeps fewer than 64 keys of the chunk for those rows.  The
    other chunks hold plenty of keys above it, so the merged lists pass the
    check and are exact.  (16 rows of one head over 16,384 keys are cut into
    chunks of 2,048 keys, sampled every 256 keys; lane group g of a row
    samples keys 4g .. 4g + 3 of each 16 of a tile.)"""
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
    the row is flagged and rescanned over all keys without a gate."""
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
