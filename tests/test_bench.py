"""bench.py: its host logic (no GPU) and, on a GPU, its one-line JSON
contract on a short run."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle import hga_oracle as O
from paper_2606_30709_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("key", ["smalllm", "train12k", "qwen32k"])
def test_gather_attend_bytes_follow_the_routed_output(key):
    """The fused gather + attention moves Q, K, V once and writes out and
    LSE; with the routed buffers written it also writes K and V of every
    valid routed row, and nothing else changes."""
    w = W.preset(key)
    e = w.elem_bytes
    rows = 1000
    on_chip = bench.algorithmic_bytes(w, rows)["gather_attend"]
    written = bench.algorithmic_bytes(w, rows, routed_out=True)["gather_attend"]
    q = w.batch * w.n_q_heads * w.seq_len * w.head_dim * e
    kv = w.batch * w.n_kv_heads * w.seq_len * w.head_dim * e
    ids = w.batch * w.n_kv_heads * w.n_chunks * w.topk_groups * 4
    assert on_chip == 2 * q + 2 * kv + w.batch * w.n_q_heads * w.seq_len * 4 + ids
    assert written - on_chip == 2 * rows * w.head_dim * e


@pytest.mark.parametrize("kw", [dict(), dict(keep_first=2, keep_last=3),
                                dict(keep_first=0, keep_last=0, force_prev=0),
                                dict(n_q_heads=4, n_kv_heads=2)])
def test_attention_flops_count_every_visible_pair(kw):
    """4*d FLOPs per (query, key) pair, the pairs counted one query at a time
    from the oracle's working set (Sec. 3.4) plus the causal current chunk."""
    w = W.preset("tiny").with_(batch=2, n_q_heads=kw.get("n_q_heads", 2),
                               n_kv_heads=kw.get("n_kv_heads", 2), seq_len=20 * 64,
                               topk_groups=5, **{k: v for k, v in kw.items()
                                                 if k not in ("n_q_heads", "n_kv_heads")})
    rng = np.random.default_rng(3)
    nc, C, G = w.n_chunks, w.chunk, w.group
    gpc = C // G
    gi = np.full((w.batch, w.n_kv_heads, nc, w.topk_groups), -1, dtype=np.int32)
    for c in range(nc):
        _, M = O.visibility(c, w.keep_first, w.keep_last, w.force_prev)
        cand = [m * gpc + t for m in M for t in range(gpc)]
        for b in range(w.batch):
            for j in range(w.n_kv_heads):
                n = min(len(cand), int(rng.integers(0, w.topk_groups + 1)))
                gi[b, j, c, :n] = np.sort(rng.choice(cand, n, replace=False)) if n else []
    pairs = 0
    for b in range(w.batch):
        for j in range(w.n_kv_heads):
            for c in range(nc):
                hist = O.working_set(c, gi[b, j, c], C, G, w.keep_first, w.keep_last,
                                     w.force_prev).size
                for t in range(C):
                    pairs += w.gqa_ratio * (hist + t + 1)
    assert bench.attention_flops(w, gi) == 4.0 * w.head_dim * pairs


@pytest.mark.gpu
def test_bench_line_contract():
    """A short run prints one JSON line with the fields the contract names,
    the roofline entry of the dominant kernel among them."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "smalllm",
                        "--steps", "3", "--warmup", "1", "--no-cpu-baseline",
                        "--settle-seconds", "0"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "routed_kv"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["higher_is_better"] is True
    assert d["config"]["workload"].startswith("smalllm")
    rf = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in rf, k
    assert rf["bound"] in ("hbm", "mfma", "alu")
    assert 0 < rf["frac"] < 1 and abs(rf["achieved"] / rf["peak"] - rf["frac"]) < 1e-3


def test_dense_causal_flops_count_every_causal_pair():
    """4*d FLOPs per (query, key) pair with key <= query, counted one pair at
    a time on a small shape."""
    w = W.preset("tiny").with_(batch=2, n_q_heads=4, n_kv_heads=2, seq_len=3 * 64)
    pairs = sum(1 for qi in range(w.seq_len) for ki in range(w.seq_len) if ki <= qi)
    assert bench.dense_causal_flops(w) == 4.0 * w.head_dim * w.batch * w.n_q_heads * pairs
