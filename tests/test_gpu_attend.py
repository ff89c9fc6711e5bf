"""GPU parity of saki_attend (reading the index's winners in RoPE space)
against the oracle's sparse_attention, through the C ABI."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from tests.parity import _bf16_ambiguity, _fp8_ambiguity

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2608_03228_amd.saki")

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _t(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV, dtype)


def _check(got, q, q_pos, keys, values, idx, extra=None):
    """|out_gpu - out_oracle| <= (2 max_j delta_j + 1e-6) * sum_j p_j |v_j| per
    element, delta_j = 1e-5 ||q|| ||k_j|| / sqrt(d) (+ extra_j): the float32
    score error of 128 products plus the float32 sin / cos of the angles."""
    want = O.sparse_attention(q, q_pos, keys, values, idx)
    d = q.shape[-1]
    for i in range(q.shape[0]):
        sel = idx[i][idx[i] >= 0]
        qr = O.rope(q[i], q_pos[i])
        kr = O.rope(keys[sel], sel)
        sc = kr @ qr / np.sqrt(d)
        p = np.exp(sc - sc.max())
        p /= p.sum()
        delta = 1e-5 * np.linalg.norm(q[i]) * np.linalg.norm(keys[sel], axis=1) / np.sqrt(d)
        if extra is not None:
            delta = delta + extra[i][: sel.size]
        bound = (2 * delta.max() + 1e-6) * (p @ np.abs(values[sel]))
        err = np.abs(got[i] - want[i])
        assert np.all(err <= bound), (i, err.max(), bound.min())


def _decode_case(N=3000, H_q=4, H_kv=1, Q=1):
    spec = W.SPECS["decode_1m"].with_(N=N, H_q=H_q, H_kv=H_kv, Q=Q)
    return W.make_layer(spec, with_values=True)


@pytest.mark.parametrize("keys_bf16", [False, True])
def test_attend_exact_keys(keys_bf16):
    """Exact keys: the sketch top-64 of each head (oracle's), a padded list,
    and causal rows with their own positions."""
    inp = _decode_case(Q=5)
    N = 3000
    keys = inp["keys"].astype(np.float32)
    if keys_bf16:
        keys = O.bf16_round(keys).astype(np.float32)
    idx = np.empty((1, 4, 5, 64), np.int32)
    for h in range(4):
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][0], 32)
        s, *_ = O.index_scores(oc["B_q"], oc["B_k"], oc["mu"], inp["queries"][0, h], keys[0, 0])
        idx[0, h] = O.topk_rows(s, O.candidate_limits(5, N), 64)
    idx[0, 1, 2, 40:] = -1  # a shorter list
    pos = np.array([2999, 2999, 100, 2500, 64], np.int32)
    out = S.saki_attend(_t(inp["values"]), _t(inp["queries"]), _t(idx, torch.int32), N,
                        keys=_t(keys, torch.bfloat16 if keys_bf16 else torch.float32),
                        q_pos=_t(pos, torch.int32)).cpu().numpy()
    out_np = S.saki_attend(_t(inp["values"]), _t(inp["queries"]), _t(idx, torch.int32), N,
                           keys=_t(keys, torch.bfloat16 if keys_bf16 else torch.float32)
                           ).cpu().numpy()
    for h in range(4):
        _check(out[0, h], inp["queries"][0, h], pos, keys[0, 0], inp["values"][0, 0], idx[0, h])
        _check(out_np[0, h], inp["queries"][0, h], np.full(5, N - 1), keys[0, 0],
               inp["values"][0, 0], idx[0, h])


@pytest.mark.parametrize("sketch,r", [("f32", 32), ("bf16", 32), ("fp8", 32), ("f32", 128),
                                      ("bf16", 16), ("bf16", 64), ("fp8", 16), ("fp8", 64),
                                      ("f32", 16)])
def test_attend_reconstructed_keys(sketch, r):
    """Keys reconstructed from the index codes: mu + B_q c (Sec. 6), rotated
    after reconstruction; the oracle reconstructs from its own codes rounded
    to the same storage, and every code may sit one storage step away."""
    inp = _decode_case(N=2000, H_q=4, H_kv=1, Q=3)
    N = 2000
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r)
    index = S.saki_build_index(_t(inp["keys"]), _t(cal["B_k"]), _t(cal["mu"]), r, sketch, 4)
    idx, _ = S.saki_score_topk(index, sketch, _t(inp["queries"]), _t(cal["B_q"]), _t(cal["mu"]),
                               1, N, N, r, k=64)
    idx = idx.cpu().numpy()  # valid lists of distinct visible keys (checked in the score tests)
    out = S.saki_attend(_t(inp["values"]), _t(inp["queries"]), _t(idx, torch.int32), N,
                        index=index, sketch=sketch, B_q=_t(cal["B_q"]), mu=_t(cal["mu"]),
                        r=r).cpu().numpy()
    rnd = {"f32": O.f32_round, "bf16": O.bf16_round, "fp8": O.fp8_round}[sketch]
    for h in range(4):
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][0], r)
        c = O.codes(oc["B_k"], oc["mu"], inp["keys"][0, 0])
        khat = O.reconstruct_keys(oc["B_q"], oc["mu"], rnd(c))
        extra = None
        if sketch != "f32":
            # a code within float32 error of a rounding midpoint may be stored
            # one step away (the rule of the score parity); its error reaches
            # the key through B_q
            amb_fn = _fp8_ambiguity if sketch == "fp8" else _bf16_ambiguity
            abs_sum = np.abs(inp["keys"][0, 0] - oc["mu"]) @ np.abs(oc["B_k"])
            amb, ulp = amb_fn(c, abs_sum)
            dk = np.linalg.norm((amb * ulp) @ np.abs(oc["B_q"]).T, axis=1)  # per key
            qn = np.linalg.norm(inp["queries"][0, h], axis=1)
            extra = np.stack([qn[i] * dk[np.maximum(idx[0, h, i], 0)] / np.sqrt(128)
                              for i in range(3)])
        _check(out[0, h], inp["queries"][0, h], np.full(3, N - 1), khat, inp["values"][0, 0],
               idx[0, h], extra)


def test_attend_full_rank_reconstruction_is_exact_attention():
    """r = d: M_d = I, so reconstructed float32 codes give the exact-key output."""
    inp = _decode_case(N=1500, H_q=2, H_kv=1, Q=2)
    N = 1500
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 128)
    index = S.saki_build_index(_t(inp["keys"]), _t(cal["B_k"]), _t(cal["mu"]), 128, "f32", 2)
    rng = np.random.default_rng(0)
    idx = np.stack([rng.choice(N, 64, replace=False) for _ in range(4)]).reshape(1, 2, 2, 64)
    idx = idx.astype(np.int32)
    a = S.saki_attend(_t(inp["values"]), _t(inp["queries"]), _t(idx, torch.int32), N,
                      index=index, sketch="f32", B_q=_t(cal["B_q"]), mu=_t(cal["mu"]),
                      r=128).cpu().numpy()
    keys = inp["keys"][0, 0].astype(np.float64)
    for h in range(2):
        # the allowance: how far float32 storage of the factors and codes moves
        # the reconstruction from the exact key (the oracle's factors, rounded)
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][0], 128)
        f = O.f32_round
        c32 = f(O.codes(f(oc["B_k"]), f(oc["mu"]), keys))
        dev = np.abs(O.reconstruct_keys(f(oc["B_q"]), f(oc["mu"]), c32) - keys)
        dk = 2.0 * np.linalg.norm(dev, axis=1)
        qn = np.linalg.norm(inp["queries"][0, h], axis=1)
        extra = np.stack([qn[i] * dk[idx[0, h, i]] / np.sqrt(128) for i in range(2)])
        _check(a[0, h], inp["queries"][0, h], np.full(2, N - 1), keys, inp["values"][0, 0],
               idx[0, h], extra)


def test_attend_sequences_groups_short_and_skipped_lists():
    """Two sequences and two KV groups; lists of 40 entries (the work-group's
    last wave has none), one of 5 (only the first wave), one empty row (zeros),
    and entries at or past N_valid (skipped); exact keys and the GQA-shared
    index's reconstruction (float32 codes)."""
    spec = W.SPECS["decode_1m"].with_(N=1200, H_q=4, H_kv=2, Q=3, batch=2)
    inp = W.make_layer(spec, with_values=True)
    N_cap, N_valid, k, G = 1200, 1100, 40, 2
    rng = np.random.default_rng(7)
    idx = np.stack([rng.choice(N_cap, k, replace=False) for _ in range(2 * 4 * 3)])
    idx = idx.reshape(2, 4, 3, k).astype(np.int32)
    idx[0, 1, 0, :] = -1   # an empty row
    idx[1, 2, 1, 5:] = -1  # five entries
    visible = np.where(idx < N_valid, idx, -1)  # what the oracle attends over
    keys, values, q = inp["keys"], inp["values"], inp["queries"]
    pos = np.full(3, N_valid - 1)
    out = S.saki_attend(_t(values), _t(q), _t(idx, torch.int32), N_valid,
                        keys=_t(keys)).cpu().numpy()
    for b in range(2):
        for h in range(4):
            g = h // G
            if b == 0 and h == 1:
                assert np.all(out[b, h, 0] == 0.0)
                rows = [1, 2]
            else:
                rows = [0, 1, 2]
            _check(out[b, h, rows], q[b, h, rows], pos[rows], keys[b, g], values[b, g],
                   visible[b, h, rows])
    # the GQA-shared index: one code set per KV head, read by its G query heads
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], 32, method="shared")
    index = S.saki_build_index(_t(keys), _t(cal["B_k"][::G]), _t(cal["mu"]), 32, "f32", 2)
    out2 = S.saki_attend(_t(values), _t(q), _t(idx, torch.int32), N_valid, index=index,
                         sketch="f32", B_q=_t(cal["B_q"]), mu=_t(cal["mu"]), r=32,
                         index_heads=2).cpu().numpy()
    assert np.all(out2[0, 1, 0] == 0.0)
    for g in range(2):
        oc = O.saki_calibrate_shared(inp["q_cal"][G * g:G * g + G], inp["k_cal"][g], 32)
        for b in range(2):
            c = O.f32_round(O.codes(oc["B_k"], oc["mu"], keys[b, g]))
            khat = O.reconstruct_keys(oc["B_q"], oc["mu"], c)
            for h in range(G * g, G * g + G):
                rows = [1, 2] if (b == 0 and h == 1) else [0, 1, 2]
                _check(out2[b, h, rows], q[b, h, rows], pos[rows], khat, values[b, g],
                       visible[b, h, rows])
