"""Seeded synthetic inputs for the SAKI retrieval-index path.

This module draws inputs only; it contains none of the index method's
arithmetic.  It follows the score model of the paper's setup section
(Sec. 3): a latent token x in R^D is projected per head to a query
q = W_Q x and a key k = W_K x, with GQA sharing of W_K between the query heads
of one KV group.  The synthetic latent stands in for the hidden states of the
real models the paper measures (LLaMA-3.1-8B, Qwen2.5-7B), whose weights and
calibration text are not available:

* x ~ N(0, diag(lambda)), lambda_i = i^-alpha (1-indexed), with ``n_out``
  outlier coordinates (drawn without replacement) whose standard deviation is
  multiplied by ``out_scale``;
* W entries are N(0, 1) times a power-law column scale i^-0.5;
* calibration uses ``T`` tokens separate from the cached sequence.

Every array is reproducible from (workload name, layer, sequence, head,
purpose, step) through ``numpy.random.SeedSequence`` spawn keys, so any subset
(one head, one layer, one step) can be regenerated on its own.  The float32
arrays returned here are *the* inputs: both the CPU oracle and the GPU library
read exactly these values.
"""
from __future__ import annotations

import dataclasses
import zlib
from dataclasses import dataclass

import numpy as np

BASE_SEED = 20260803
_PURPOSE = {"wq": 1, "wk": 2, "outliers": 3, "calib": 4, "keys": 5, "queries": 6, "wv": 7}
_CHUNK = 65536  # rows drawn per call, fixed so that prefixes stay identical


@dataclass(frozen=True)
class WorkloadSpec:
    """Shape and spectrum of one synthetic workload.

    ``Q`` is the number of query rows per (sequence, head) and per decode step.
    With ``causal`` the queries are the sequence's own positions
    ``q_start .. N-1`` and row i may see keys j <= position_i; otherwise the
    queries are fresh tokens and see all N keys.
    """

    name: str
    H_q: int
    H_kv: int
    d: int
    D: int
    alpha: float
    n_out: int
    out_scale: float
    T: int
    N: int
    Q: int
    causal: bool
    q_start: int = 0
    batch: int = 1
    layers: int = 1
    steps: int = 1
    ranks: tuple = (32,)
    sketches: tuple = ("f32",)

    def with_(self, **kw) -> "WorkloadSpec":
        """Same seeds (same name), other sizes: prefixes of every stream agree."""
        return dataclasses.replace(self, **kw)


SPECS = {
    # One head, d=128, latent 256, N=1024 keys, 256 fresh queries, no mask.
    "single_head_d128": WorkloadSpec(
        "single_head_d128", H_q=1, H_kv=1, d=128, D=256, alpha=1.0, n_out=4,
        out_scale=20.0, T=512, N=1024, Q=256, causal=False, ranks=(32,),
        sketches=("f32",)),
    # One LLaMA-3.1-8B-shaped layer: 32 query heads on 8 KV heads, causal
    # self-queries at positions 64..4095.
    "llama31_8b_layer": WorkloadSpec(
        "llama31_8b_layer", H_q=32, H_kv=8, d=128, D=512, alpha=1.0, n_out=4,
        out_scale=20.0, T=512, N=4096, Q=4096 - 64, causal=True, q_start=64,
        ranks=(16, 32, 64), sketches=("f32", "bf16")),
    # All 32 layers of the same shape.
    "llama31_8b_sweep": WorkloadSpec(
        "llama31_8b_sweep", H_q=32, H_kv=8, d=128, D=512, alpha=1.0, n_out=4,
        out_scale=20.0, T=512, N=4096, Q=4096 - 64, causal=True, q_start=64,
        layers=32, ranks=(16, 32, 64), sketches=("bf16",)),
    # Long-context decode: 2^20 cached keys per KV head, one query per head
    # per step.
    "decode_1m": WorkloadSpec(
        "decode_1m", H_q=32, H_kv=8, d=128, D=512, alpha=1.0, n_out=4,
        out_scale=20.0, T=512, N=1 << 20, Q=1, causal=False, steps=64,
        ranks=(32,), sketches=("bf16",)),
    # Qwen2.5-7B-shaped batched decode: 28 layers, 28 query heads on 4 KV
    # heads, 8 sequences of 131072 keys, 16 queries per head per step.
    "qwen25_7b_decode": WorkloadSpec(
        "qwen25_7b_decode", H_q=28, H_kv=4, d=128, D=512, alpha=0.7, n_out=8,
        out_scale=50.0, T=512, N=131072, Q=16, causal=False, batch=8,
        layers=28, steps=8, ranks=(32,), sketches=("bf16",)),
}


def rng(spec: WorkloadSpec, purpose: str, layer: int = 0, seq: int = 0,
        head: int = 0, step: int = 0) -> np.random.Generator:
    """Independent PCG64 stream keyed by (workload, layer, seq, head, purpose, step)."""
    key = (zlib.crc32(spec.name.encode()), layer, seq, head, _PURPOSE[purpose], step)
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence(BASE_SEED, spawn_key=key)))


def latent_std(spec: WorkloadSpec, layer: int = 0) -> np.ndarray:
    """Per-coordinate standard deviation of the latent token (float64 [D])."""
    i = np.arange(1, spec.D + 1, dtype=np.float64)
    std = np.sqrt(i ** (-spec.alpha))
    out = rng(spec, "outliers", layer).choice(spec.D, size=spec.n_out, replace=False)
    std[out] *= spec.out_scale
    return std


def weights(spec: WorkloadSpec, layer: int = 0):
    """W_Q [H_q, d, D] and W_K [H_kv, d, D] (float64)."""
    col = np.arange(1, spec.D + 1, dtype=np.float64) ** -0.5
    wq = np.stack([rng(spec, "wq", layer, head=h).standard_normal((spec.d, spec.D)) * col
                   for h in range(spec.H_q)])
    wk = np.stack([rng(spec, "wk", layer, head=g).standard_normal((spec.d, spec.D)) * col
                   for g in range(spec.H_kv)])
    return wq, wk


def value_weights(spec: WorkloadSpec, layer: int = 0):
    """W_V [H_kv, d, D] (float64), drawn like W_K."""
    col = np.arange(1, spec.D + 1, dtype=np.float64) ** -0.5
    return np.stack([rng(spec, "wv", layer, head=g).standard_normal((spec.d, spec.D)) * col
                     for g in range(spec.H_kv)])


def tokens(spec: WorkloadSpec, purpose: str, n: int, layer: int = 0, seq: int = 0,
           step: int = 0) -> np.ndarray:
    """n latent tokens [n, D] (float64), drawn in fixed-size chunks."""
    g = rng(spec, purpose, layer, seq=seq, step=step)
    std = latent_std(spec, layer)
    out = np.empty((n, spec.D), np.float64)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        out[s:e] = g.standard_normal((e - s, spec.D)) * std
    return out


def _project(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """[n, D] x [H, d, D] -> [H, n, d] float32, computed in float64 by chunks."""
    H, d, _ = w.shape
    out = np.empty((H, x.shape[0], d), np.float32)
    for s in range(0, x.shape[0], _CHUNK):
        e = min(x.shape[0], s + _CHUNK)
        for h in range(H):
            out[h, s:e] = x[s:e] @ w[h].T
    return out


def make_layer(spec: WorkloadSpec, layer: int = 0, seqs=None, step: int = 0,
               with_calib: bool = True, with_values: bool = False) -> dict:
    """All inputs of one layer.

    Returns a dict with
      q_cal [H_q, T, d] f32, k_cal [H_kv, T, d] f32 (calibration tokens),
      keys [B, H_kv, N, d] f32, queries [B, H_q, Q, d] f32,
      q_pos int32 [Q] (causal) or None, W_Q [H_q, d, D] and W_K [H_kv, d, D]
      (float64, for the weight-SVD baseline); with_values also
      values [B, H_kv, N, d] f32 = W_V x of the same cached tokens.
    ``seqs`` selects which sequences of the batch to build (default all).
    """
    seqs = list(range(spec.batch)) if seqs is None else list(seqs)
    wq, wk = weights(spec, layer)
    out = {"W_Q": wq, "W_K": wk, "spec": spec, "layer": layer, "step": step}
    if with_calib:
        xc = tokens(spec, "calib", spec.T, layer)
        out["q_cal"] = _project(xc, wq)
        out["k_cal"] = _project(xc, wk)
    keys = np.empty((len(seqs), spec.H_kv, spec.N, spec.d), np.float32)
    queries = np.empty((len(seqs), spec.H_q, spec.Q, spec.d), np.float32)
    if with_values:
        wv = value_weights(spec, layer)
        out["values"] = np.empty((len(seqs), spec.H_kv, spec.N, spec.d), np.float32)
    for bi, s in enumerate(seqs):
        xs = tokens(spec, "keys", spec.N, layer, seq=s)
        keys[bi] = _project(xs, wk)
        if with_values:
            out["values"][bi] = _project(xs, wv)
        if spec.causal:
            queries[bi] = _project(xs[spec.q_start:spec.q_start + spec.Q], wq)
        else:
            xq = tokens(spec, "queries", spec.Q, layer, seq=s, step=step)
            queries[bi] = _project(xq, wq)
    out["keys"] = keys
    out["queries"] = queries
    out["q_pos"] = (np.arange(spec.q_start, spec.q_start + spec.Q, dtype=np.int32)
                    if spec.causal else None)
    return out
