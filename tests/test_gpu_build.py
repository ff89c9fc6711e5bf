"""GPU parity of the key-code build (Eq. 4) over key ranges that cut the
work-group slices at odd places: every rank, float32 and bf16 keys, every
code type, against the oracle's float64 codes, with the codes outside the
range left untouched.

The build forms float32 products on the bf16 MFMA from three bf16 terms per
operand; its codes must stay within AMBIG_REL of their absolute-value sum,
the float32 error bound the bf16 parity rule assumes."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from tests.parity import AMBIG_REL

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2608_03228_amd.saki")

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _t(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV, dtype)


def _inputs(N, B, H_q, H_kv, r, seed):
    spec = W.SPECS["llama31_8b_layer"].with_(N=N, Q=1, q_start=0, H_q=H_q, H_kv=H_kv, batch=B)
    keys = W.make_layer(spec, with_calib=False)["keys"]
    rng = np.random.default_rng(seed)
    B_k = (rng.standard_normal((H_q, 128, r)) / np.sqrt(128)).astype(np.float32)
    mu = (rng.standard_normal((H_kv, 128)) * 0.3).astype(np.float32)
    return keys, B_k, mu


def _check(got, keys64, B_k, mu, sketch, G):
    """got [B, H_q, n, r] exported codes of keys64 [B, H_kv, n, d]."""
    for b in range(got.shape[0]):
        for h in range(got.shape[1]):
            x = keys64[b, h // G] - mu[h // G].astype(np.float64)
            w = B_k[h].astype(np.float64)
            exact = x @ w
            scale = np.abs(x) @ np.abs(w)
            g = got[b, h].astype(np.float64)
            if sketch == "f32":
                assert np.max(np.abs(g - exact) / scale) < AMBIG_REL, (b, h)
            elif sketch == "bf16":
                assert np.all(O.bf16_round(g) == g)
                ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(exact), 1e-30))) - 7)
                assert np.all(np.abs(g - exact) <= 0.5 * ulp + AMBIG_REL * scale), (b, h)
            else:
                assert np.all(O.fp8_round(g) == g)
                mag = np.maximum(np.abs(exact), 1e-30)
                ulp = np.where(mag < 2.0 ** -6, 2.0 ** -9, np.exp2(np.floor(np.log2(mag)) - 3))
                assert np.all(np.abs(g - exact) <= 0.5 * ulp + AMBIG_REL * scale), (b, h)


@pytest.mark.parametrize("r", [16, 32, 64, 128])
@pytest.mark.parametrize("key_dtype", ["f32", "bf16"])
def test_build_range_across_slices(r, key_dtype):
    """20,000 keys of two KV heads (several work-group slices per head), a
    range starting and ending off every 16- and 32-key boundary; f32, bf16
    and fp8 codes."""
    B, H_q, H_kv, N = 2, 8, 2, 20_000
    keys, B_k, mu = _inputs(N, B, H_q, H_kv, r, seed=r)
    kt = _t(keys, torch.bfloat16 if key_dtype == "bf16" else torch.float32)
    keys64 = kt.float().cpu().numpy().astype(np.float64)  # the keys the GPU reads
    n0, n1 = 1237, 1237 + 15_001
    for sketch in ("f32", "bf16", "fp8"):
        nb = S.saki_index_bytes(B, H_q, N, r, sketch)
        index = torch.full((nb,), 0x3C, dtype=torch.uint8, device=DEV)  # a marker pattern
        before = S.saki_index_export(index, sketch, B, H_q, N, r).cpu().numpy()
        S.saki_build_index(kt, _t(B_k), _t(mu), r, sketch, H_q, index=index, n_begin=n0,
                           n_count=n1 - n0)
        torch.cuda.synchronize()
        got = S.saki_index_export(index, sketch, B, H_q, N, r).cpu().numpy()
        _check(got[:, :, n0:n1], keys64[:, :, n0:n1], B_k, mu, sketch, H_q // H_kv)
        # codes outside the range are untouched
        np.testing.assert_array_equal(got[:, :, :n0], before[:, :, :n0])
        np.testing.assert_array_equal(got[:, :, n1:], before[:, :, n1:])


def test_short_ranges_one_head_per_work_group():
    """Ranges of at most 256 keys take one query head per work-group: odd
    starts and lengths, the last key of the cache, and one key."""
    B, H_q, H_kv, N, r = 1, 8, 2, 5_000, 32
    keys, B_k, mu = _inputs(N, B, H_q, H_kv, r, seed=5)
    kt = _t(keys)
    keys64 = keys.astype(np.float64)
    nb = S.saki_index_bytes(B, H_q, N, r, "f32")
    for n0, cnt in ((0, 1), (17, 239), (4_093, 256), (4_999, 1), (2_048, 33)):
        index = torch.full((nb,), 0x3C, dtype=torch.uint8, device=DEV)
        before = S.saki_index_export(index, "f32", B, H_q, N, r).cpu().numpy()
        S.saki_build_index(kt, _t(B_k), _t(mu), r, "f32", H_q, index=index, n_begin=n0, n_count=cnt)
        torch.cuda.synchronize()
        got = S.saki_index_export(index, "f32", B, H_q, N, r).cpu().numpy()
        _check(got[:, :, n0:n0 + cnt], keys64[:, :, n0:n0 + cnt], B_k, mu, "f32", H_q // H_kv)
        np.testing.assert_array_equal(got[:, :, :n0], before[:, :, :n0])
        np.testing.assert_array_equal(got[:, :, n0 + cnt:], before[:, :, n0 + cnt:])
