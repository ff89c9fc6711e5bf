"""CPU checks of bench.py's contract: the one-GPU refusal, the pair count of
the headline workload, the score stage's algorithmic work, and the lookup
of the profiled HBM traffic by kernel-source digest."""
import json
import os
import subprocess
import sys

import bench
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _sweep():
    s = W.SPECS["llama31_8b_sweep"]
    return s.with_(H_q=s.H_q * s.layers, H_kv=s.H_kv * s.layers), s.N


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "exactly one GPU" in json.loads(p.stdout.strip().splitlines()[-1])["error"]


def test_sweep_pair_count_is_the_causal_sum():
    spec, N = _sweep()
    # rows at positions 64 .. 4095 see keys 0 .. position: sum of 65 .. 4096
    per_head = sum(range(65, 4097))
    assert spec.H_q == 1024 and spec.q_start == 64 and spec.Q == 4032 and N == 4096
    assert bench.candidates(spec, N) == per_head * 1024 == 8_589_901_824


def test_score_stage_work_is_2r_flops_per_pair():
    spec, N = _sweep()
    t = bench.roofline_terms(spec, 32, "bf16", 64)["score_topk"]
    assert t["flops"] == 2 * 32 * bench.candidates(spec, N)
    assert t["flop_unit"] == "bf16" and t["peak_flops"] == 2516.6


def test_profiled_traffic_follows_the_kernel_source(monkeypatch):
    """A row counts only for the kernel source it was measured on."""
    inst = "score_batch_kernel<32, 1>"
    row = next(ln for ln in open(bench.TRAFFIC_FILE).read().splitlines()
               if ln.startswith("| score_batch_kernel | llama31_8b_sweep |"))
    cells = [c.strip() for c in row.strip().strip("|").split("|")]
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: cells[2])
    assert bench.measured_traffic("score_batch_kernel", "llama31_8b_sweep", inst) == float(cells[5])
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 16)
    assert bench.measured_traffic("score_batch_kernel", "llama31_8b_sweep", inst) is None
