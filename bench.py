"""Benchmark of the SAKI retrieval-index path on one MI355X.

Headline workload: all 32 LLaMA-3.1-8B-shaped layers as the 1,024 query
heads (256 KV heads) of one launch of each kernel: d = 128, N = 4096 cached
keys, causal query rows at positions 64..4095, rank-32 bf16 sketches.  One
step is one pass of the whole path over that batch:

  1. calibrate   float64 moments of the 512 calibration tokens on the GPU (side
                 stream, for the next batch, after the score stage enqueued
                 before it), copied back; host float64 factorisation into
                 B_q, B_k, mu; factors uploaded
  2. build       key codes for every query head
  3. score_topk  query sketches, sketch scores and the top-64 per (query, head)
  4. recall      exact float64 q.k top-64 and hits against the sketch top-64
                 (enqueued in the next step ahead of its build: the host
                 factorisation outlasts a step's GPU work, and the GPU's wait
                 for it then precedes the evaluation, not the build and score;
                 every timed step runs one recall, the first of them the last
                 warm-up batch's, and the last batch's runs after timing)

Inputs (keys, queries, positions, calibration tokens) are resident in HBM
before timing starts.  `value` is the metric's unit of work, (query, allowed
key) pairs scored and top-64-selected, divided by the score_topk stage's
HIP-event time; `ms_per_step` is the whole step.  The same run also reports
(key `extra`) the long-context decode workload over 2^20 keys (64 steps),
one layer-step of the Qwen2.5-7B-shaped batched decode, the single-head
recall table (SAKI, span variants, key PCA, weight SVD) and the single
LLaMA-shaped layer in float32 and bf16 at r = 16, 32, 64.
Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "keys scored+top-64 selected/sec; % of HBM / MFMA roofline; recall@64"
PEAK = {"hbm_GBps": 8000.0, "bf16_TFLOPs": 2516.6, "fp32_TFLOPs": 157.3, "fp64_TFLOPs": 78.6}
ES = {"f32": 4, "bf16": 2, "fp8": 1}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llama31_8b_sweep")
    ap.add_argument("--r", type=int, default=32)
    ap.add_argument("--sketch", default="bf16", choices=["bf16", "f32", "fp8"])
    ap.add_argument("--k", type=int, default=64)
    ap.add_argument("--shared", action="store_true",
                    help="GQA-shared index: one code set per KV head (pooled query moment)")
    ap.add_argument("--method", default="opt", choices=["opt", "sap_map", "sap_svd", "key_pca"],
                    help="factors of the batched workloads: the paper's optimum, its span "
                         "variants (Sec. 6) or the key-PCA baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="only the selected workload (profiling runs)")
    ap.add_argument("--no-attend", action="store_true",
                    help="decode: leave out reading the winners (RoPE attention over the top-64)")
    ap.add_argument("--decode-steps", type=int, default=64,
                    help="timed steps of the long-context decode workload in the extras")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter scale) and exit")
    return ap.parse_args()


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------ traffic

# the kernel that dominates each stage, and the template instance launched
# for (r, sketch) as rocprofv3 names it
STAGE_KERNEL = {"build": "build_index_kernel", "score_topk": "score_batch_kernel",
                "recall": "exact_gate_kernel"}
STAGE_INSTANCE = {
    "build": lambda r, sk: f"build_index_kernel<{r}, false, {({'f32': 0, 'bf16': 1, 'fp8': 2})[sk]}>",
    "score_topk": lambda r, sk: f"score_batch_kernel<{r}, {({'f32': 0, 'bf16': 1, 'fp8': 2})[sk]}>",
    "recall": lambda r, sk: "exact_gate_kernel<false>",
}
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_03228_amd", "csrc", "saki_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.md")


def kernel_source_digest():
    import hashlib
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel, workload, instance):
    """HBM bytes per step of `kernel`'s launches on `workload` (the one-pass
    scan launches twice per step) from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (scaled by a plain copy of known size), or None when
    no row matches the current kernel source and the template instance the
    run launches."""
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    digest = kernel_source_digest()
    for ln in lines:
        cells = [c.strip() for c in ln.strip().strip("|").split("|")]
        if (len(cells) >= 7 and cells[0] == kernel and cells[1] == workload and cells[2] == digest
                and cells[6].startswith(f"`{instance}`")):
            try:
                return float(cells[5])
            except ValueError:
                return None
    return None


def copy_probe(nbytes):
    """A plain device-to-device copy of known size (the scale for the HBM
    byte counters): prints bytes read and written per launch."""
    import torch
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe": {"read_bytes": n * 4, "write_bytes": n * 4, "launches": 5}}))


# ------------------------------------------------------------------ work counts

def candidates(spec, N_valid):
    """Number of (query, allowed key) pairs in one step (all heads, sequences)."""
    if spec.causal:
        pos = np.arange(spec.q_start, spec.q_start + spec.Q, dtype=np.int64)
        per_head = int(np.minimum(pos + 1, N_valid).sum())
    else:
        per_head = spec.Q * N_valid
    return per_head * spec.H_q * spec.batch


def roofline_terms(spec, r, sketch, k):
    """Algorithmic work per launch of each batched stage (bytes moved at least
    once, flops of the defined arithmetic counted once)."""
    es = ES[sketch]
    rows = spec.batch * spec.H_q * spec.Q
    pairs = candidates(spec, spec.N)
    heads = spec.batch * spec.H_q
    return {
        # 2 r flops per causal pair; codes read once per head, queries read
        # once, top-k (idx + score) written once
        "score_topk": {"bytes": heads * spec.N * r * es + rows * spec.d * 4 + rows * k * 8,
                       "flops": 2 * r * pairs,
                       "peak_flops": PEAK["fp32_TFLOPs"] if sketch == "f32" else PEAK["bf16_TFLOPs"],
                       "flop_unit": "fp32" if sketch == "f32" else "bf16"},
        # keys read once per KV head, codes written once per query head
        "build": {"bytes": spec.batch * spec.H_kv * spec.N * spec.d * 4 + heads * spec.N * r * es,
                  "flops": 2 * spec.d * r * spec.N * heads,
                  "peak_flops": PEAK["fp32_TFLOPs"], "flop_unit": "fp32"},
        # keys and queries read once, lists read, hits written; 2 d flops per
        # pair counted once, priced at the bf16 peak of its hi/lo products
        "recall": {"bytes": spec.batch * spec.H_kv * spec.N * spec.d * 4 + rows * spec.d * 4
                   + rows * k * 4 + rows * 4,
                   "flops": 2 * spec.d * pairs,
                   "peak_flops": PEAK["bf16_TFLOPs"], "flop_unit": "bf16"},
    }


def stage_roofline(term, ms):
    s = ms / 1e3
    return {"ms": ms, "GB/s": term["bytes"] / s / 1e9, "TFLOP/s": term["flops"] / s / 1e12,
            "frac_hbm": term["bytes"] / s / 1e9 / PEAK["hbm_GBps"],
            "frac_flops": term["flops"] / s / 1e12 / term["peak_flops"],
            "flop_dtype": term["flop_unit"]}


# ------------------------------------------------------------------ inputs

def layers_as_heads(spec):
    """All layers of a workload as the heads of one layer (layer l's query
    head h is head l * H_q + h, its KV head g is l * H_kv + g), so that one
    launch of each kernel covers every head of the model."""
    import workloads as W
    layers = [W.make_layer(spec, layer=l) for l in range(spec.layers)]
    inp = {"spec": spec.with_(H_q=spec.H_q * spec.layers, H_kv=spec.H_kv * spec.layers, layers=1),
           "q_pos": layers[0]["q_pos"], "n_layers": spec.layers}
    for n, ax in (("q_cal", 0), ("k_cal", 0), ("keys", 1), ("queries", 1)):
        inp[n] = np.concatenate([x[n] for x in layers], axis=ax)
    return inp


def decode_queries(spec, step):
    """The fresh query tokens of one decode step, [B, H_q, Q, d] float32."""
    import workloads as W
    wq, _ = W.weights(spec)
    out = np.empty((spec.batch, spec.H_q, spec.Q, spec.d), np.float32)
    for b in range(spec.batch):
        out[b] = W._project(W.tokens(spec, "queries", spec.Q, seq=b, step=step), wq)
    return out


# ------------------------------------------------------------------ CPU baseline

def _cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, r, sketch, k, heads, heads_1t):
    """The oracle, as it stands, on a bounded sample of the workload: the
    metric's unit of work (sketch scores and the top-k of every query row,
    float64 numpy) for the query heads `heads` at all host BLAS threads, and
    for `heads_1t` at one thread.  Calibration and the exact recall are not
    part of the unit and are not timed."""
    import oracle as O
    from threadpoolctl import threadpool_info, threadpool_limits
    spec = inp["spec"]
    G = spec.H_q // spec.H_kv
    lim = O.candidate_limits(spec.Q, spec.N, inp["q_pos"])
    facs = {}
    for h in sorted(set(heads) | set(heads_1t)):
        oc = O.saki_calibrate(inp["q_cal"][h], inp["k_cal"][h // G], r)
        facs[h] = (oc["B_q"], oc["B_k"], oc["mu"])

    def unit(sample):
        t0 = time.perf_counter()
        n = 0
        for h in sample:
            Bq, Bk, mu = facs[h]
            s_hat, *_ = O.index_scores(Bq, Bk, mu, inp["queries"][0, h], inp["keys"][0, h // G],
                                       sketch)
            O.topk_rows(s_hat, lim, k)
            n += int(lim.sum())
        return n, time.perf_counter() - t0

    all_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    n_all, t_all = unit(heads)
    with threadpool_limits(1):
        n_one, t_one = unit(heads_1t)
    return {"value": n_all / t_all, "unit": "keys/s", "cores": int(all_threads), "kind": "oracle",
            "value_1_thread": n_one / t_one,
            "sample": f"sketch scores + top-{k} ({sketch} codes emulated, float64 numpy) of all "
                      f"{spec.Q} query rows of {len(heads)} query heads {list(heads)} "
                      f"({n_all} pairs, {t_all:.1f} s at {all_threads} BLAS threads), and of "
                      f"heads {list(heads_1t)} at 1 thread ({n_one} pairs, {t_one:.1f} s); "
                      f"host {_cpu_model()}, os.cpu_count()={os.cpu_count()}"}


# ------------------------------------------------------------------ batched workloads

def run_batched(inp, r, sk, k, steps, warmup, method="opt"):
    """Time `steps` steps (after `warmup`) of the batched path on inputs
    already resident in HBM; returns the measurements as a dict."""
    import torch
    from paper_2608_03228_amd import saki as S
    dev = torch.device("cuda:0")
    spec = inp["spec"]
    keys = torch.from_numpy(inp["keys"]).to(dev)
    q = torch.from_numpy(inp["queries"]).to(dev)
    pos = torch.from_numpy(inp["q_pos"]).to(dev) if inp["q_pos"] is not None else None
    B, H_kv, N, d = keys.shape
    H_q = spec.H_q
    # device buffers allocated once, reused by every step
    index = torch.empty(S.saki_index_bytes(B, H_q, N, r, sk), dtype=torch.uint8, device=dev)
    ws = torch.empty(max(1, S.saki_score_topk_workspace_bytes(B, H_q, spec.Q, N, r, k, sk)),
                     dtype=torch.uint8, device=dev)
    wsr = torch.empty(max(1, S.saki_recall_workspace_bytes(B, H_q, H_kv, spec.Q, N, d, k)),
                      dtype=torch.uint8, device=dev)
    top_idx = torch.empty((B, H_q, spec.Q, k), dtype=torch.int32, device=dev)
    top_sc = torch.empty((B, H_q, spec.Q, k), dtype=torch.float32, device=dev)
    hits = torch.empty((B, H_q, spec.Q), dtype=torch.int32, device=dev)
    # the factors live in one flat buffer (one upload per step); f_dev are views
    f_shape = {"B_q": (H_q, d, r), "B_k": (H_q, d, r), "mu": (H_kv, d)}
    f_off, f_total = {}, 0
    for n, sh in f_shape.items():
        f_off[n] = (f_total, f_total + int(np.prod(sh)))
        f_total = f_off[n][1]
    f_flat = torch.empty(f_total, dtype=torch.float32, device=dev)
    f_dev = {n: f_flat[a:b].view(f_shape[n]) for n, (a, b) in f_off.items()}
    # calibration: float64 moments on the GPU (side stream, default priority),
    # copied to pinned host memory; the host factorises them while the GPU
    # still runs the previous batch
    q_cal = torch.from_numpy(inp["q_cal"]).to(dev)
    k_cal = torch.from_numpy(inp["k_cal"]).to(dev)
    side = torch.cuda.Stream()
    m_shape = {"Sq": (H_q, d, d), "Sk": (H_kv, d, d), "mu": (H_kv, d)}
    m_dev = [{n: torch.empty(sh, dtype=torch.float64, device=dev) for n, sh in m_shape.items()}
             for _ in range(2)]
    m_host = [{n: torch.empty(sh, dtype=torch.float64).pin_memory() for n, sh in m_shape.items()}
              for _ in range(2)]
    m_done = [None, None]
    side.wait_stream(torch.cuda.current_stream())  # calibration tokens uploaded
    score_done = [None]  # the last score stage enqueued on the launch stream

    def enqueue_moments(sl):
        with torch.cuda.stream(side):
            # after the score stage enqueued last: the moments then run while
            # the GPU waits for the host factorisation, never beside a build
            # or score
            if score_done[0] is not None:
                side.wait_event(score_done[0])
            S.saki_calibration_moments(q_cal, k_cal, m_dev[sl]["Sq"], m_dev[sl]["Sk"],
                                       m_dev[sl]["mu"], stream=side)
            for n in m_shape:
                m_host[sl][n].copy_(m_dev[sl][n], non_blocking=True)
            m_done[sl] = torch.cuda.Event()
            m_done[sl].record(side)

    def factorise(sl, out=None):
        h = m_host[sl]
        return S.saki_calibrate_from_moments(h["Sq"].numpy(), h["Sk"].numpy(), h["mu"].numpy(),
                                             r, method=method, with_sigma=False, out=out)
    # two pinned staging slots: the host calibrates batch i+1 while the GPU
    # still works on batch i, writing the factors straight into the slot
    slots = [torch.empty(f_total, dtype=torch.float32).pin_memory() for _ in range(2)]
    slot_out = [{n: slots[i].numpy()[a:b].reshape(f_shape[n]) for n, (a, b) in f_off.items()}
                for i in range(2)]
    slot_done = [None, None]
    ev, ev_recall = [], []
    n_step = [0]
    pending = [False]  # a batch scored whose recall is not enqueued yet
    enqueue_moments(0)

    def recall(timed_stages):
        # the evaluation of the batch scored last (its top-64 lists)
        if timed_stages:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record()
        S.saki_recall(keys, q, top_idx, N, q_pos=pos, k=k, ws=wsr, hits=hits,
                      want_exact=False)
        if timed_stages:
            e[1].record()
            ev_recall.append(e)
        pending[0] = False

    def step(timed_stages=True):
        sl = n_step[0] % 2
        n_step[0] += 1
        m_done[sl].synchronize()
        enqueue_moments(1 - sl)  # the next batch's moments overlap this one
        if slot_done[sl] is not None:
            slot_done[sl].synchronize()
        factorise(sl, out=slot_out[sl])
        f_flat.copy_(slots[sl], non_blocking=True)
        slot_done[sl] = torch.cuda.Event()
        slot_done[sl].record()
        # the previous batch's recall goes first: the host factorisation runs a
        # little longer than a step's GPU work, and the GPU's wait for it then
        # falls before the evaluation kernel, not before the build and score
        if pending[0]:
            recall(timed_stages)
        if timed_stages:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record()
        S.saki_build_index(keys, f_dev["B_k"], f_dev["mu"], r, sk, H_q, index=index)
        if timed_stages:
            e[1].record()
        S.saki_score_topk(index, sk, q, f_dev["B_q"], f_dev["mu"], H_kv, N, N, r, q_pos=pos,
                          k=k, ws=ws, top_idx=top_idx, top_score=top_sc)
        if timed_stages:
            e[2].record()
            ev.append(e)
        score_done[0] = torch.cuda.Event()
        score_done[0].record()
        pending[0] = True

    for _ in range(warmup):
        step(timed_stages=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        # each timed step runs one recall (of the batch before it: the first
        # one evaluates the last warm-up batch), one build and one score
        step()  # stage events on the launch stream, inside the timed region
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    # the last batch's evaluation, after the timed region (its time is used
    # only when no timed step ran a recall: no warm-up and one step)
    recall(not ev_recall)
    torch.cuda.synchronize()
    names = ["build", "score_topk", "recall"]
    stage_ms = {n: float(np.mean([es[i].elapsed_time(es[i + 1]) for es in ev]))
                for i, n in enumerate(names[:2])}
    stage_ms["recall"] = float(np.mean([es[0].elapsed_time(es[1]) for es in ev_recall]))
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    e[0].record(side)
    with torch.cuda.stream(side):
        S.saki_calibration_moments(q_cal, k_cal, m_dev[0]["Sq"], m_dev[0]["Sk"], m_dev[0]["mu"],
                                   stream=side)
    e[1].record(side)
    torch.cuda.synchronize()
    stage_ms["calibrate_moments_gpu"] = e[0].elapsed_time(e[1])
    t_cal = time.perf_counter()
    for _ in range(3):
        factorise(0)
    stage_ms["calibrate_factorise_host"] = (time.perf_counter() - t_cal) / 3 * 1e3

    h = hits.cpu().numpy().astype(np.int64)
    per_head = h.sum(axis=(0, 2)) / (k * spec.Q)
    last512 = h[:, :, -512:].sum(axis=(0, 2)) / (k * min(512, spec.Q))
    pairs = candidates(spec, N)
    terms = roofline_terms(spec, r, sk, k)
    return {
        "pairs": pairs, "ms_per_step": dt * 1e3, "stages_ms": stage_ms,
        "value": pairs / (stage_ms["score_topk"] / 1e3),
        "stage_rooflines": {n: stage_roofline(terms[n], stage_ms[n]) for n in names},
        "terms": terms,
        "recall_at_64": {"median_over_heads": float(np.median(per_head)),
                         "mean_over_heads": float(np.mean(per_head)),
                         "last512_median": float(np.median(last512)),
                         "hits_total": int(h.sum()), "rows": int(h.size)},
    }


def score_roofline(res, spec, r, sk, k, method):
    """The headline roofline: the score_topk stage (score_batch_kernel
    dominates it), 2 r flops per allowed pair against the sketch dtype's MFMA
    peak."""
    t = res["terms"]["score_topk"]
    sec = res["stages_ms"]["score_topk"] / 1e3
    roof = {"bound": "mfma", "achieved": t["flops"] / sec / 1e12, "peak": t["peak_flops"],
            "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = (measured_traffic(STAGE_KERNEL["score_topk"], spec.name,
                                        STAGE_INSTANCE["score_topk"](r, sk))
                       if method == "opt" and k == 64 else None)
    roof["kernel"] = "score_topk"
    roof["work"] = {"flops": t["flops"], "flop_dtype": t["flop_unit"], "bytes": t["bytes"],
                    "pairs": res["pairs"], "flops_per_pair": 2 * r}
    return roof


# ------------------------------------------------------------------ decode workloads

def run_decode(spec, r, sk, k, steps, warmup, shared=False, attend=True, cpu=False):
    """Long-context decode: the index of N cached keys is built once; a step
    appends the newest key's codes and scores every head's fresh queries
    against all N codes with a top-k per row (then, with `attend`, RoPE
    attention over each row's top-k).  Exact recall of every step is
    evaluated after the timed loop.  Returns the measurements as a dict."""
    import torch
    import workloads as W
    from paper_2608_03228_amd import saki as S
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    inp = W.make_layer(spec, with_values=attend)
    t_gen = time.perf_counter() - t_gen
    keys = torch.from_numpy(inp["keys"]).to(dev)
    values = torch.from_numpy(inp.pop("values")).to(dev) if attend else None
    B, H_kv, N, d = keys.shape
    H_q, Q = spec.H_q, spec.Q
    n_q = warmup + steps
    qs = torch.from_numpy(np.stack([decode_queries(spec, s) for s in range(n_q)])).to(dev)
    G = H_q // H_kv
    IH = H_kv if shared else H_q  # code sets per sequence
    cal = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r, method="shared" if shared else "opt")
    Bq, Bk, mu = (torch.from_numpy(cal[n]).to(dev) for n in ("B_q", "B_k", "mu"))
    if shared:
        Bk = Bk[::G].contiguous()
    index = torch.empty(S.saki_index_bytes(B, IH, N, r, sk), dtype=torch.uint8, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    S.saki_build_index(keys, Bk, mu, r, sk, IH, index=index)
    e1.record()
    torch.cuda.synchronize()
    build_full_ms = e0.elapsed_time(e1)
    ws = torch.empty(max(1, S.saki_score_topk_workspace_bytes(B, H_q, Q, N, r, k, sk, IH)),
                     dtype=torch.uint8, device=dev)
    top_idx = torch.empty((n_q, B, H_q, Q, k), dtype=torch.int32, device=dev)
    top_sc = torch.empty((n_q, B, H_q, Q, k), dtype=torch.float32, device=dev)
    att_out = torch.empty((B, H_q, Q, d), dtype=torch.float32, device=dev)
    ev = []

    def step(s, timed=False):
        if timed:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            e[0].record()
        S.saki_build_index(keys, Bk, mu, r, sk, IH, index=index, n_begin=N - 1, n_count=1)
        if timed:
            e[1].record()
        S.saki_score_topk(index, sk, qs[s], Bq, mu, H_kv, N, N, r, k=k, ws=ws,
                          top_idx=top_idx[s], top_score=top_sc[s], index_heads=IH)
        if timed:
            e[2].record()
        if attend:  # read the winners: exact keys and values, RoPE, softmax
            S.saki_attend(values, qs[s], top_idx[s], N, keys=keys, out=att_out)
        if timed:
            e[3].record()
            ev.append(e)

    for s in range(warmup):
        step(s)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(warmup, n_q):
        step(s, timed=True)  # stage events on the launch stream, inside the timed region
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    append_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    score_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    attend_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))

    # exact recall of every step (evaluation, outside the timed loop)
    wsr = torch.empty(max(1, S.saki_recall_workspace_bytes(B, H_q, H_kv, Q, N, d, k)),
                      dtype=torch.uint8, device=dev)
    hits = torch.empty((n_q, B, H_q, Q), dtype=torch.int32, device=dev)
    e0.record()
    for s in range(n_q):
        S.saki_recall(keys, qs[s], top_idx[s], N, k=k, ws=wsr, hits=hits[s], want_exact=False)
    e1.record()
    torch.cuda.synchronize()
    recall_ms = e0.elapsed_time(e1) / n_q
    h = hits.cpu().numpy().astype(np.int64)
    per_head = h.sum(axis=(0, 1, 3)) / (k * Q * n_q * B)  # over steps, sequences, queries

    code_bytes = B * IH * N * r * ES[sk]
    scan_bytes = code_bytes + B * H_q * Q * d * 4 + B * H_q * Q * k * 8
    roof = {"bound": "hbm", "achieved": scan_bytes / (score_ms / 1e3) / 1e9,
            "peak": PEAK["hbm_GBps"], "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    # the kernel the library runs for this shape: 16 or more queries per head
    # take the MFMA kernels (one pass over the codes from 16,384 keys on),
    # fewer the streaming kernel with 1 or 4 rows per wave
    st = {"f32": 0, "bf16": 1, "fp8": 2}[sk]
    if Q >= 16:
        kern = "score_scan_kernel" if N >= 16384 else "score_batch_kernel"
        inst = f"{kern}<{r}, {st}>"
    else:
        kern = "score_stream_kernel"
        inst = f"{kern}<{r}, {st}, {4 if (H_q // IH) * Q >= 4 else 1}>"
    roof["traffic"] = measured_traffic(kern, spec.name, inst)
    roof["kernel"] = "score_topk"
    roof["work"] = {"bytes": scan_bytes, "code_bytes": code_bytes}

    cpu_res = None
    if cpu:  # the oracle on one head of one step
        import oracle as O
        oc = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], r)
        q0 = decode_queries(spec, warmup)[0, 0]
        t = time.perf_counter()
        s_hat, *_ = O.index_scores(oc["B_q"], oc["B_k"], oc["mu"], q0, inp["keys"][0, 0], sk)
        O.topk_rows(s_hat, O.candidate_limits(Q, N), k)
        dtc = time.perf_counter() - t
        cpu_res = {"value": Q * N / dtc, "unit": "keys/s", "cores": os.cpu_count(),
                   "kind": "oracle",
                   "sample": f"query head 0 of one step ({Q * N} keys): codes+scores+top-{k} "
                             f"in float64 numpy; {dtc:.1f} s; host {_cpu_model()}"}
    return {
        "value": B * H_q * Q * N / (score_ms / 1e3), "unit": "keys/s",
        "ms_per_step": dt * 1e3, "steps": steps, "warmup": warmup,
        "config": {"workload": spec.name, "H_q": H_q, "H_kv": H_kv, "d": d,
                   "latent_D": spec.D, "N": N, "queries_per_head": Q, "batch": B, "r": r,
                   "sketch": sk, "k": k, "index": "gqa_shared" if shared else "per_query_head",
                   "step": "append one key + score + top-64" +
                           (" + RoPE attention over the top-64" if attend else "") +
                           " (index built once)"},
        "roofline": roof, "cpu_baseline": cpu_res,
        "stages_ms": {"append": append_ms, "score_topk": score_ms,
                      "attend_top64": attend_ms if attend else None,
                      "build_full_once": build_full_ms, "recall_eval": recall_ms,
                      "input_generation_ms": t_gen * 1e3},
        "recall_at_64": {"median_over_heads": float(np.median(per_head)),
                         "mean_over_heads": float(np.mean(per_head)),
                         "hits_total": int(h.sum()), "rows": int(h.size)},
    }


# ------------------------------------------------------------------ extras

def recall_table_single_head(r=32, k=64):
    """The single-head workload (1 head, N = 1024, 256 fresh queries, fp32
    sketches): recall@64 of SAKI, its span variants, key PCA and weight SVD,
    each run through the same GPU kernels with its own factors."""
    import torch
    import workloads as W
    from paper_2608_03228_amd import saki as S
    dev = torch.device("cuda:0")
    spec = W.SPECS["single_head_d128"]
    inp = W.make_layer(spec)
    keys = torch.from_numpy(inp["keys"]).to(dev)
    q = torch.from_numpy(inp["queries"]).to(dev)
    N = spec.N
    pca = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r, method="key_pca")
    facs = {}
    for name, method in (("saki", "opt"), ("sap_map", "sap_map"), ("sap_svd", "sap_svd"),
                         ("key_pca", "key_pca")):
        c = S.saki_calibrate(inp["q_cal"], inp["k_cal"], r, method=method)
        facs[name] = (c["B_q"], c["B_k"], c["mu"])
    wq, wk = S.saki_weight_svd_factors(inp["W_K"], 1, r)
    facs["weight_svd"] = (wq, wk, pca["mu"])
    out = {}
    for name, (Bq, Bk, mu) in facs.items():
        Bq_t, Bk_t, mu_t = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (Bq, Bk, mu))
        index = S.saki_build_index(keys, Bk_t, mu_t, r, "f32", 1)
        idx, _ = S.saki_score_topk(index, "f32", q, Bq_t, mu_t, 1, N, N, r, k=k)
        hits, _ = S.saki_recall(keys, q, idx, N, k=k, want_exact=False)
        h = int(hits.sum().item())
        out[name] = {"recall_at_64": round(h / (k * spec.Q), 4), "hits": h}
    return {"workload": spec.name, "r": r, "sketch": "f32", "rows": spec.Q, "table": out}


def layer_variants(steps, warmup, k=64):
    """The single LLaMA-shaped layer in float32 and bf16 sketches at r = 16,
    32, 64: score_topk throughput and its fraction of the dtype's MFMA peak."""
    import workloads as W
    spec = W.SPECS["llama31_8b_layer"]
    inp = W.make_layer(spec)
    out = {}
    for sk in ("f32", "bf16"):
        for r in (16, 32, 64):
            res = run_batched(inp, r, sk, k, steps, warmup)
            sr = res["stage_rooflines"]["score_topk"]
            out[f"{sk}_r{r}"] = {"value": res["value"], "unit": "keys/s",
                                 "score_topk_ms": res["stages_ms"]["score_topk"],
                                 "score_TFLOPs": sr["TFLOP/s"], "score_frac_mfma": sr["frac_flops"],
                                 "mfma_peak_dtype": sr["flop_dtype"],
                                 "ms_per_step": res["ms_per_step"],
                                 "recall_median": res["recall_at_64"]["median_over_heads"]}
    return out


def _decode_summary(res):
    return {"value": res["value"], "unit": res["unit"], "ms_per_step": res["ms_per_step"],
            "steps": res["steps"], "config": res["config"],
            "score_topk_ms": res["stages_ms"]["score_topk"],
            "score_frac_hbm": res["roofline"]["frac"], "roofline": res["roofline"],
            "stages_ms": res["stages_ms"], "recall_at_64": res["recall_at_64"]}


# ------------------------------------------------------------------ main

def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on exactly one GPU; --gpus must be 1 "
                                   "(multi-GPU sharding is described in the design notes)"}))
        sys.exit(2)
    if args.copy_probe:
        return copy_probe(args.copy_probe)
    import workloads as W

    spec = W.SPECS[args.workload]
    r, sk, k = args.r, args.sketch, args.k
    if spec.steps > 1 and not spec.causal:  # decode workloads on their own
        res = run_decode(spec, r, sk, k, args.steps, args.warmup, shared=args.shared,
                         attend=not args.no_attend, cpu=not args.no_cpu_baseline)
        out = {"metric": METRIC, "value": res["value"], "unit": "keys/s", "n_gpus": 1,
               "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
               "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": sk,
               "data": "synthetic", "config": res["config"], "roofline": res["roofline"],
               "cpu_baseline": res["cpu_baseline"], "stages_ms": res["stages_ms"],
               "recall_at_64": res["recall_at_64"]}
        print(json.dumps(out), flush=True)
        return
    if spec.batch != 1 or spec.steps != 1:
        raise SystemExit(f"the batched step runs one sequence and one step; {args.workload} is not")

    log(f"generating {spec.name}")
    t_gen = time.perf_counter()
    inp = W.make_layer(spec) if spec.layers == 1 else layers_as_heads(spec)
    t_gen = time.perf_counter() - t_gen
    log(f"timing {spec.name} ({t_gen:.1f} s of input generation)")
    res = run_batched(inp, r, sk, k, args.steps, args.warmup, method=args.method)
    bspec = inp["spec"]
    roof = score_roofline(res, bspec, r, sk, k, args.method)
    log(f"score_topk {res['stages_ms']['score_topk']:.3f} ms, {roof['frac']:.4f} of peak")

    cpu = None
    if not args.no_cpu_baseline:
        log("CPU baseline")
        # every third query head of layers 0, 15 and 31 of the sweep (of the
        # one layer otherwise); the first eight of them at one thread
        layers = (0, 15, 31) if inp.get("n_layers", 1) == 32 else (0,)
        heads = [l * spec.H_q + h for l in layers for h in range(0, spec.H_q, 3)]
        cpu = cpu_baseline(inp, r, sk, k, heads, heads[:8])
    del inp

    extra = {}
    if not args.no_extra:
        log("extra: single-head recall table")
        extra["single_head_d128_recall"] = recall_table_single_head()
        log("extra: LLaMA-shaped layer variants")
        extra["llama31_8b_layer"] = layer_variants(5, 2, k)
        log("extra: decode over 2^20 keys")
        extra["decode_1m"] = _decode_summary(
            run_decode(W.SPECS["decode_1m"], 32, "bf16", k, args.decode_steps, 3))
        log("extra: Qwen-shaped decode layer")
        extra["qwen25_7b_decode"] = _decode_summary(
            run_decode(W.SPECS["qwen25_7b_decode"], 32, "bf16", k, 8, 2, attend=False))

    out = {
        "metric": METRIC, "value": res["value"], "unit": "keys/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": sk,
        "data": "synthetic",
        "config": {"workload": spec.name, "layers_as_heads": spec.layers,
                   "H_q": bspec.H_q, "H_kv": bspec.H_kv, "d": bspec.d, "latent_D": bspec.D,
                   "N": bspec.N, "queries_per_head": bspec.Q, "causal": bspec.causal, "r": r,
                   "sketch": sk, "k": k, "calib_tokens": bspec.T, "factors": args.method,
                   "pairs_per_step": res["pairs"],
                   "value_basis": "pairs / score_topk stage time (HIP events)",
                   "step": "calibrate (GPU moments + host factors) + build + score_topk + "
                           "recall"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stages_ms": res["stages_ms"],
        "stage_rooflines": res["stage_rooflines"],
        "value_whole_step": res["pairs"] / (res["ms_per_step"] / 1e3),
        "recall_at_64": res["recall_at_64"],
        "input_generation_s": t_gen,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
