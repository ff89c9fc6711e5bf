"""GPU test of saki_score_topk_noalloc, the score entry point that allocates
nothing (its split-key workspace is the library's static scratch array),
against saki_score_topk with a caller-owned workspace, through the C ABI.
Two calls in a row per shape, the second smaller, so the second reads a
scratch array that still holds the first call's contents."""
import numpy as np
import pytest

import workloads as W
from tests.test_gpu_parity import _t, check_head

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2608_03228_amd.saki")

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _score_both(inp, r, sketch, N_valid, q_pos=None):
    """The same index scored by both entry points; returns numpy (idx, score)
    pairs and the inputs the oracle check needs."""
    spec = inp["spec"]
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r)
    keys, q = _t(inp["keys"]), _t(inp["queries"])
    B_q, B_k, mu = _t(cal["B_q"]), _t(cal["B_k"]), _t(cal["mu"])
    B, H_kv, N_cap, _ = keys.shape
    H_q, Q = spec.H_q, spec.Q
    pos = _t(q_pos, torch.int32) if q_pos is not None else None
    index = S.saki_build_index(keys, B_k, mu, r, sketch, H_q)
    need = S.saki_score_topk_workspace_bytes(B, H_q, Q, N_valid, r, 64, sketch)
    assert 256 < need <= S.saki_noalloc_scratch_bytes()  # the shape uses the scratch array
    ref = S.saki_score_topk(index, sketch, q, B_q, mu, H_kv, N_cap, N_valid, r, q_pos=pos)
    idx = torch.full((B, H_q, Q, 64), -7, dtype=torch.int32, device=DEV)
    sc = torch.full((B, H_q, Q, 64), 7.0, dtype=torch.float32, device=DEV)
    S.saki_score_topk_noalloc(index, sketch, q, B_q, mu, H_kv, N_cap, N_valid, r, idx, sc,
                              q_pos=pos)
    torch.cuda.synchronize()
    return (ref[0].cpu().numpy(), ref[1].cpu().numpy()), (idx.cpu().numpy(), sc.cpu().numpy()), cal


@pytest.mark.parametrize("first,second", [
    # decode rows: the key axis of every row split into chunks (partial lists)
    (dict(N=200_000, Q=1, H_q=8, H_kv=2), dict(N=50_000, Q=1, H_q=4, H_kv=1)),
    # 16 queries per head over long rows: the one-pass scan with chunk gates
    # and redo flags
    (dict(N=40_003, Q=16, H_q=2, H_kv=1), dict(N=17_000, Q=16, H_q=2, H_kv=1)),
    # 16 or more queries per head over fewer than 16,384 keys: the two-pass
    # scorer, whose query sketches (and, past 4,096 keys, partial lists) live
    # in the scratch array
    (dict(N=5_000, Q=64, H_q=8, H_kv=2), dict(N=3_000, Q=32, H_q=4, H_kv=1)),
])
def test_noalloc_equals_workspace_entry_point(first, second):
    for shape, sketch in ((first, "bf16"), (second, "f32")):
        spec = W.SPECS["decode_1m"].with_(**shape)
        inp = W.make_layer(spec)
        (ri, rs), (gi, gs), _ = _score_both(inp, 32, sketch, spec.N)
        np.testing.assert_array_equal(gi, ri)
        np.testing.assert_array_equal(gs, rs)
        # and the oracle's parity rule on two heads
        out = {"idx": gi, "score": gs}
        mode = "bf16_emul" if sketch == "bf16" else "f32"
        for h in (0, spec.H_q - 1):
            n, ex, diff = check_head(inp, out, 0, h, 32, mode)
            assert diff == 0, (shape, h, ex, diff)


def test_noalloc_rejects_calls_beyond_its_scratch():
    """A call whose workspace exceeds the static array fails with
    SAKI_ERR_WORKSPACE before anything is launched."""
    H = 2047
    need = S.saki_score_topk_workspace_bytes(1, H, 16, 16_384, 32, 64, "bf16")
    assert need > S.saki_noalloc_scratch_bytes()
    index = torch.empty(S.saki_index_bytes(1, H, 16_384, 32, "bf16"), dtype=torch.uint8,
                        device=DEV)
    q = torch.zeros((1, H, 16, 128), dtype=torch.float32, device=DEV)
    B_q = torch.zeros((H, 128, 32), dtype=torch.float32, device=DEV)
    mu = torch.zeros((1, 128), dtype=torch.float32, device=DEV)
    idx = torch.empty((1, H, 16, 64), dtype=torch.int32, device=DEV)
    with pytest.raises(S.SakiError) as e:
        S.saki_score_topk_noalloc(index, "bf16", q, B_q, mu, 1, 16_384, 16_384, 32, idx)
    assert e.value.status == -3
