#!/usr/bin/env python3
"""Routed-attention throughput of one layer on one MI355X.

One step = the whole hot path over one batch of synthetic input: chunk and
group summaries, chunk routing, group refinement, gather of the routed K/V,
and exact attention (inputs already resident in HBM).  By default a step is
three C-ABI calls: hga_build_summaries_qbar (summaries and the routing query
means in one launch), hga_route_qbar (chunk and group selection) and
hga_gather_attend (the attention gathers each routed group's rows from the
resident K/V straight into its LDS tiles; with --routed-out it also writes
them to the routed buffers, the standalone gather's output).
--route fused / separate use hga_route or the two routing calls instead,
--gather separate uses hga_gather_kv + hga_attend (identical results).  The
default workload is the largest single-GPU prefill, the Qwen3-30B-A3B
attention-layer shape (B1, 32 query heads over 4 KV heads, d128, 32768
tokens, bf16, RoPE base 1e6, C64 G16, first chunk and the 2 most recent
chunks hot, K_c 30, K_g 48 -> 3.125% of the context fetched by the last
chunk); --workload selects another preset.

Prints one JSON line.  The step rate comes from the wall clock between two
synchronizations around the timed steps.  In about ten of the timed steps,
spread evenly over them, the dominant kernel (the attention) is launched with
a pair of HIP events that its dispatch records at the kernel's own start and
end on the launch stream; its algorithmic bytes (or FLOPs, above the ridge
point) over the mean duration give the roofline entry.  A second pass with
events between all calls gives the per-stage breakdown of the other kernels.
The float64 oracle timed on the host cores over a bounded sample of the same
workload gives the CPU baseline.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak
VALU_FP32_PEAK_TFLOPS = 157.3   # fp32 vector peak (256 CUs at 2.4 GHz)

ROUTE_STAGES = {
    "qbar": ("build_summaries_qbar", "route_qbar"),
    "fused": ("build_summaries", "route"),
    "separate": ("build_summaries", "route_chunks", "route_groups"),
}
GATHER_STAGES = {
    "fused": ("gather_attend",),
    "separate": ("gather_kv", "attend"),
}
ATTENTION_STAGES = ("attend", "gather_attend")


def algorithmic_bytes(w, n_valid_rows: int, routed_out: bool = False) -> dict:
    """Bytes each kernel must move at least once per step (compulsory
    traffic).  n_valid_rows = routed token rows (all heads, all chunks);
    routed_out: the fused gather + attention also writes the routed rows."""
    B, Hq, Hkv, d, N, C, G = (w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.seq_len,
                              w.chunk, w.group)
    e = w.elem_bytes
    nc = w.n_chunks
    gpc = C // G
    kv_tok = B * Hkv * N * d * e          # one of K or V
    q_tok = B * Hq * N * d * e
    table_c = B * Hkv * nc * d * 4
    table_g = B * Hkv * nc * gpc * d * 4
    routed = n_valid_rows * d * e         # one of K or V
    return {
        "build_summaries": kv_tok + table_c + table_g,
        "route_chunks": q_tok + table_c + table_c + B * Hkv * nc * w.topk_chunks * 4,
        "route_groups": table_c + table_g + B * Hkv * nc * (w.topk_chunks + w.topk_groups) * 4,
        "route": (q_tok + 2 * table_c + table_g +
                  B * Hkv * nc * (w.topk_chunks + w.topk_groups) * 4),
        "build_summaries_qbar": kv_tok + table_c + table_g + q_tok + table_c,
        "route_qbar": 2 * table_c + table_g + B * Hkv * nc * (w.topk_chunks + w.topk_groups) * 4,
        "gather_kv": 4 * routed + B * Hkv * nc * w.topk_groups * 4,
        "attend": q_tok + 2 * kv_tok + 2 * routed + q_tok + B * Hq * N * 4,
        # the routed rows are rows of the resident K/V, which is read once
        # as a whole (every chunk is some unit's current chunk); with
        # routed_out they are written once to the routed buffers and never
        # read back
        "gather_attend": (q_tok + 2 * kv_tok + q_tok + B * Hq * N * 4 +
                          (2 * routed if routed_out else 0) +
                          B * Hkv * nc * w.topk_groups * 4),
    }


def _prefill_label(w) -> str:
    return (f"B{w.batch} H{w.n_q_heads}/{w.n_kv_heads} d{w.head_dim} N{w.seq_len} {w.dtype} "
            f"C{w.chunk} G{w.group} F{w.keep_first} L{w.keep_last} Kc{w.topk_chunks} "
            f"Kg{w.topk_groups}")


def attention_flops(w, group_idx: np.ndarray) -> float:
    """Exact-attention FLOPs of a step: 4*d per (query, key) pair (QK^T and PV)."""
    C, G, d, r = w.chunk, w.group, w.head_dim, w.gqa_ratio
    F, W = w.keep_first, max(w.keep_last, 1 if w.force_prev else 0)
    valid = (group_idx >= 0).sum(axis=-1)             # [B, Hkv, nq]
    pairs = 0
    for i in range(group_idx.shape[2]):
        c = w.q_chunk0 + i
        a = min(F, c)
        nd = a + (c - max(a, max(0, c - W)))
        hist = nd * C
        pairs += r * (C * hist * group_idx.shape[0] * group_idx.shape[1]
                      + C * G * int(valid[:, :, i].sum()) + group_idx.shape[0] *
                      group_idx.shape[1] * C * (C + 1) // 2)
    return 4.0 * d * pairs


ATTEND_SOURCES = ("attend_mfma.hip", "attend_common.hpp", "hga_device.hpp", "hga_internal.hpp")


def traffic_file(kernel: str, workload_key: str) -> str:
    return os.path.join(ROOT, "profiles", f"{kernel}_{workload_key}_traffic.txt")
COPY_BYTES = 256 << 20


def attend_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in ATTEND_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_30709_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload_key: str, routed_out: bool = False):
    """HBM bytes per launch of the attention kernel (`kernel`: attend or
    gather_attend, the latter with or without the routed-buffer writes) from
    the committed counter summary, or None when there is none, it covers the
    other form, or the kernel source changed since the counters were taken."""
    try:
        vals = {}
        with open(traffic_file(kernel, workload_key)) as f:
            for line in f:
                if "=" in line and not line.lstrip().startswith("#"):
                    k, v = (x.strip() for x in line.split("=", 1))
                    vals[k] = v
        if vals.get("kernel_source_sha256") != attend_source_hash():
            return None
        if vals.get("workload") != workload_key:
            return None
        if kernel == "gather_attend" and vals.get("routed_out") != str(int(routed_out)):
            return None
        return int(float(vals["traffic_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


def probe_traffic(w, inp, gather_mode: str, routed_out: bool):
    """For counter collection: the pipeline once, the attention call 5 times
    (hga_gather_attend, with or without the routed-buffer writes, or
    hga_attend with gather_mode "separate"), then 5 plain device copies of
    COPY_BYTES (the calibration for FETCH_SIZE and WRITE_SIZE)."""
    import torch

    from paper_2606_30709_amd.pipeline import PrefillPipeline
    pipe = PrefillPipeline(w, inp, gather_mode=gather_mode, routed_out=routed_out)
    pipe.step()
    for _ in range(5):
        if gather_mode == "fused":
            pipe.gather_attend()
        else:
            pipe.attend()
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"probe": "traffic", "workload": w.key, "copy_bytes": COPY_BYTES,
                      "kernel": "gather_attend" if gather_mode == "fused" else "attend",
                      "routed_out": int(pipe.routed_out),
                      "kernel_source_sha256": attend_source_hash()}), flush=True)


def cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def _spread_order(n: int) -> list:
    """0 .. n-1 in bit-reversed order of the next power of two (any prefix is
    spread over the whole range)."""
    bits = max(1, (n - 1).bit_length())
    rev = [int(format(i, f"0{bits}b")[::-1], 2) for i in range(1 << bits)]
    return [i for i in rev if i < n]


def cpu_baseline(w, inp, max_seconds: float, block_chunks: int = 64) -> dict:
    """The float64 oracle, as it stands, over a bounded sample of the same
    workload: pieces of `block_chunks` query chunks of one (batch, KV head),
    all five stages for those query chunks (summaries of every chunk up to
    the piece's end, routing, gather, attention), taken with the blocks in a
    spread-out order and the units in turn, until max_seconds of CPU work.
    A piece is worth block_chunks * chunk / n_kv_heads tokens of the layer."""
    from threadpoolctl import threadpool_info

    from oracle import hga_oracle as O
    from paper_2606_30709_amd import workloads as W

    r, C = w.gqa_ratio, w.chunk
    units = [(b, j) for b in range(w.batch) for j in range(w.n_kv_heads)]
    n_blocks = (w.n_chunks + block_chunks - 1) // block_chunks
    pieces = [(u, blk) for blk in _spread_order(n_blocks) for u in units]
    done = chunks = 0
    t0 = time.perf_counter()
    while True:
        (b, j), blk = pieces[done % len(pieces)]
        c0 = blk * block_chunks
        c1 = min(w.n_chunks, c0 + block_chunks)
        q = W.storage_to_f64(inp["q"][b:b + 1, j * r:(j + 1) * r, c0 * C:c1 * C], w.dtype)
        k = W.storage_to_f64(inp["k"][b:b + 1, j:j + 1, :c1 * C], w.dtype)
        v = W.storage_to_f64(inp["v"][b:b + 1, j:j + 1, :c1 * C], w.dtype)
        O.hga_forward(q, k, v, chunk=C, group=w.group, keep_first=w.keep_first,
                      keep_last=w.keep_last, force_prev=w.force_prev, topk_chunks=w.topk_chunks,
                      topk_groups=w.topk_groups, rope_base=w.rope_base, q_chunk0=c0,
                      with_gather=True)
        done += 1
        chunks += c1 - c0
        if time.perf_counter() - t0 > max_seconds:
            break
    dt = time.perf_counter() - t0
    tokens = chunks * C / w.n_kv_heads
    threads = 1
    for pool in threadpool_info():
        threads = max(threads, int(pool.get("num_threads", 1)))
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} pieces of {block_chunks} query chunks of one (batch, KV head) "
                      f"({chunks} unit-chunks, {chunks / (w.n_chunks * len(units)):.2f} of the "
                      f"layer's {w.n_chunks * len(units)}: the {len(pieces)} pieces in turn, "
                      f"blocks spread over the sequence), five stages, float64 NumPy, "
                      f"{dt:.1f} s",
            "cpu": cpu_model(), "host_cpus": os.cpu_count()}


def settle(step, seconds: float) -> int:
    """Run `step` untimed, in batches of ten with a synchronization after
    each, until `seconds` of wall time have passed (before the warm-up
    steps): the GPU's clocks reach their steady state first, so a short timed
    region does not measure the ramp.  Returns the steps run."""
    import torch
    n = 0
    t_end = time.perf_counter() + seconds
    while time.perf_counter() < t_end:
        for _ in range(10):
            step()
        n += 10
        torch.cuda.synchronize()
    return n


def measured_h2d_bandwidth(sizes=(1 << 20, 64 << 20), reps: int = 20) -> dict:
    """GB/s of plain host-to-device copies from pinned host memory (the
    reference for the host-link gathers), per size in bytes: the mean over
    `reps` copies timed with events on the current stream."""
    import torch
    out = {}
    for n in sizes:
        src = torch.empty(n, dtype=torch.uint8, pin_memory=True)
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        for _ in range(3):
            dst.copy_(src, non_blocking=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            dst.copy_(src, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        out[f"{n >> 20}MiB"] = round(n * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    return out


def measured_copy_bandwidth(nbytes: int = 1 << 30, reps: int = 10) -> float:
    """Achievable HBM bandwidth on this device: GB/s of a streaming copy of
    nbytes (each byte read once and written once), well beyond the 256 MB
    Infinity Cache.  torch's vectorized elementwise kernel (x * 1 over fp32)
    is used: it streams faster here than the runtime's blit copy."""
    import torch
    src = torch.zeros(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) * 1e-3 / reps
    del src, dst
    torch.cuda.empty_cache()
    return 2 * nbytes / sec / 1e9


def dense_causal_flops(w) -> float:
    """FLOPs of dense causal attention over the workload's Q/K/V: 4*d per
    visible (query, key) pair (two d-long products, a multiply and an add
    each), N(N+1)/2 pairs per query head."""
    return 4.0 * w.head_dim * w.batch * w.n_q_heads * w.seq_len * (w.seq_len + 1) / 2


def dense_comparator(w, pipe, reps: int = 20):
    """Dense causal attention over the same Q/K/V with PyTorch's fused SDPA
    (a comparator only: flash or memory-efficient kernels, never the
    unfused math path), or None where no fused kernel is available."""
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel

    q, k, v = pipe.q, pipe.k, pipe.v
    if w.n_q_heads != w.n_kv_heads:
        r = w.gqa_ratio
        k = k.repeat_interleave(r, dim=1)
        v = v.repeat_interleave(r, dim=1)
    try:
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            out = F.scaled_dot_product_attention(q, k, v, is_causal=True)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                out = F.scaled_dot_product_attention(q, k, v, is_causal=True)
            e1.record()
            torch.cuda.synchronize()
    except RuntimeError as e:
        return {"available": False, "reason": str(e).splitlines()[0][:200]}
    ms = e0.elapsed_time(e1) / reps
    del out
    tflops = dense_causal_flops(w) / (ms * 1e-3) / 1e12
    out = {"available": True, "kernel": "torch SDPA (flash / memory-efficient), causal",
           "ms": round(ms, 4), "tokens_per_s": round(w.batch * w.seq_len / (ms * 1e-3), 1),
           "TFLOP_s": round(tflops, 1)}
    if w.dtype == "bf16":
        out["mfma_frac"] = round(tflops / MFMA_BF16_PEAK_TFLOPS, 4)
    return out


def decode_bench(w, inp, args):
    """The 64-token decode block: route, gather of the routed groups from the
    pinned host history, attention, append; one block per step."""
    import torch

    from paper_2606_30709_amd.pipeline import DecodePipeline
    pipe = DecodePipeline(w, inp, qbar_first=not args.route_from_q)
    for _ in range(args.warmup):
        pipe.step()
    torch.cuda.synchronize()
    K = args.steps
    t0 = time.perf_counter()
    for _ in range(K):
        pipe.step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / K
    pcie = pipe.pcie_bytes_per_step()
    res = {
        "metric": "routed-attn decode tokens/s (64-token block)",
        "value": round(w.chunk * w.batch / dt, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": (f"{w.key}: decode block B{w.batch} H{w.n_q_heads}/{w.n_kv_heads} "
                                f"d{w.head_dim} position {w.q_chunk0 * w.chunk} {w.dtype} "
                                f"F{w.keep_first} L{w.keep_last} Kc{w.topk_chunks} "
                                f"Kg{w.topk_groups}, history in pinned host memory"),
                   "seed": inp["seed"]},
        "pcie_bytes_per_block": pcie,
        "pcie_gbs_at_block_rate": round(pcie / dt / 1e9, 2),
        "pcie_measured_GB_s": measured_h2d_bandwidth(),
    }
    print(json.dumps(res), flush=True)


def decode_sequence_bench(w, inp, args):
    """Consecutive 64-token decode blocks (the last w.decode_blocks chunks):
    per block route, gather of the routed groups (through the warm LRU cache
    unless --no-cache, else straight from pinned host memory), split
    attention, append.  One step = the whole sequence of blocks, starting
    from an empty cache (a fresh sequence); the uncached rate is measured
    in the same run for comparison."""
    import torch

    from paper_2606_30709_amd.pipeline import DecodeSequencePipeline
    slots = args.cache_slots or 8 * w.topk_groups

    schedule = "serial" if args.route_from_q else args.schedule
    slots_or_none = None if args.no_cache else slots

    def run(cache_slots, sched):
        pipe = DecodeSequencePipeline(w, inp, cache_slots=cache_slots,
                                      qbar_first=not args.route_from_q)
        overlapped = sched.endswith("overlapped")
        step = pipe.step_overlapped if overlapped else pipe.step
        if sched.startswith("graph"):
            step = pipe.capture(overlapped).replay
        for _ in range(args.warmup):
            pipe.reset_cache()
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            pipe.reset_cache()
            step()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        routed = int((pipe.group_idx >= 0).sum().item())
        return dt, pipe.pcie_bytes(), routed

    dt, pcie, routed = run(slots_or_none, schedule)
    descr = {
        "serial": "route, gather, attend per block on one stream",
        "overlapped": "gather of block b+1 on a second stream while block b attends",
        "graph-serial": "the one-stream schedule replayed as a HIP graph",
        "graph-overlapped": ("gather of block b+1 on a second stream while block b attends, "
                             "the step replayed as a HIP graph (stream joins as graph edges)"),
    }
    res = {
        "metric": "routed-attn decode tokens/s (64-token blocks in sequence)",
        "value": round(w.chunk * w.batch * w.decode_blocks / dt, 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": (f"{w.key}: {w.decode_blocks} consecutive decode blocks "
                                f"B{w.batch} H{w.n_q_heads}/{w.n_kv_heads} d{w.head_dim} from "
                                f"position {w.q_chunk0 * w.chunk} {w.dtype} F{w.keep_first} "
                                f"L{w.keep_last} Kc{w.topk_chunks} Kg{w.topk_groups}, history "
                                f"in pinned host memory"),
                   "seed": inp["seed"],
                   "warm_cache_slots_per_head": None if args.no_cache else slots},
        "schedule": f"{schedule}: {descr[schedule]}",
        "us_per_block": round(dt * 1e6 / w.decode_blocks, 2),
        "pcie_bytes_per_block": pcie // w.decode_blocks,
        "pcie_measured_GB_s": measured_h2d_bandwidth(),
        "routed_groups_fetched_from_host": round(
            pcie / (2 * w.group * w.head_dim * w.elem_bytes) / max(routed, 1), 4),
    }
    if not args.route_from_q:
        res["other_schedules_us_per_block"] = {
            sc: round(run(slots_or_none, sc)[0] * 1e6 / w.decode_blocks, 2)
            for sc in descr if sc != schedule}
    if not args.no_cache:
        dt0, pcie0, _ = run(None, schedule)
        res["uncached"] = {"us_per_block": round(dt0 * 1e6 / w.decode_blocks, 2),
                           "pcie_bytes_per_block": pcie0 // w.decode_blocks}
    print(json.dumps(res), flush=True)


def backward_bench(w, inp, args):
    """The attention backward (hga_attend_backward) of a prefill preset: after
    one forward step, each timed step zeroes dk, dv and computes dq, dk, dv
    for a fixed output gradient.  Roofline: 10*d FLOP per (query, key) pair
    (S recomputed, dP, dQ, dK, dV) against the bf16 matrix-core peak."""
    import torch

    from paper_2606_30709_amd.pipeline import PrefillPipeline
    pipe = PrefillPipeline(w, inp)
    pipe.step()
    torch.cuda.synchronize()
    gen = np.random.default_rng(w.seed + 99)
    dout = torch.from_numpy(gen.standard_normal(pipe.q.shape).astype(np.float32)).to(
        torch.bfloat16).cuda()
    for _ in range(args.warmup):
        pipe.backward(dout)
    torch.cuda.synchronize()
    K = args.steps
    t0 = time.perf_counter()
    for _ in range(K):
        pipe.backward(dout)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / K
    # the kernel alone, between events (allocation and zeroing outside)
    from paper_2606_30709_amd import hga
    dq = torch.empty(pipe.q.shape, dtype=torch.float32, device="cuda")
    dk = torch.zeros(pipe.k.shape, dtype=torch.float32, device="cuda")
    dv = torch.zeros_like(dk)
    times = []
    for _ in range(max(5, K // 4)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        hga.hga_attend_backward(pipe.plan, pipe.q, 0, pipe.k, pipe.v, pipe.group_idx, pipe.out,
                                pipe.lse, dout, dq, dk, dv)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3)
    ksec = float(np.median(times))
    flops = 2.5 * attention_flops(w, pipe.group_idx.cpu().numpy())
    res = {
        "metric": "routed-attn backward tokens/s per layer",
        "value": round(w.batch * w.seq_len / dt, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.key}: attention backward " + _prefill_label(w),
                   "seed": inp["seed"]},
        "kernel_us": round(ksec * 1e6, 2),
        "roofline": {"bound": "mfma", "achieved": round(flops / ksec / 1e12, 2),
                     "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(flops / ksec / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                     "alg_flops_per_launch": flops, "traffic": None},
    }
    print(json.dumps(res), flush=True)


def blockwise_bench(w, inp, args):
    """The prompt as a sequence of 64-token blocks (hga_prefill_blocks: per
    block, routing against the chunks closed so far, gather + attention,
    then the append of the block's summaries); one step = the whole prompt."""
    import torch

    from paper_2606_30709_amd.pipeline import BlockPrefillPipeline
    split = not args.block_exact
    pipe = BlockPrefillPipeline(w, inp, split_attend=split)
    for _ in range(args.warmup):
        pipe.step()
    torch.cuda.synchronize()
    K = args.steps
    t0 = time.perf_counter()
    for _ in range(K):
        pipe.step()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / K
    tokens = w.batch * w.seq_len
    res = {
        "metric": "routed-attn block-sequential prefill tokens/s",
        "value": round(tokens / dt, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": (f"{w.key}: block-sequential prefill B{w.batch} "
                                f"H{w.n_q_heads}/{w.n_kv_heads} d{w.head_dim} N{w.seq_len} "
                                f"{w.dtype}, {w.n_chunks} blocks of {w.chunk} tokens"),
                   "seed": inp["seed"]},
        "us_per_block": round(dt * 1e6 / w.n_chunks, 2),
        "attention": "split (hga_gather_attend_split)" if split else "hga_gather_attend",
        "launches_per_block": 4 if split else 3,
    }
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen32k",
                    help="workload preset (default qwen32k, the largest single-GPU prefill: "
                         "the Qwen3-30B-A3B attention-layer shape)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="CPU budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--settle-seconds", type=float, default=0.3,
                    help="untimed steps before the warm-up steps, until this much wall time "
                         "has passed (clocks at their steady state)")
    ap.add_argument("--dense", action="store_true",
                    help="also time dense causal attention (torch SDPA) on the same Q/K/V; "
                         "on by default for train12k")
    ap.add_argument("--route", choices=("qbar", "fused", "separate"), default="qbar",
                    help="qbar: hga_build_summaries_qbar + hga_route_qbar; fused: "
                         "hga_build_summaries + hga_route; separate: hga_build_summaries + "
                         "hga_route_chunks + hga_route_groups (identical results)")
    ap.add_argument("--gather", choices=("fused", "separate"), default="fused",
                    help="fused: hga_gather_attend (the attention stages the routed rows from "
                         "the resident K/V); separate: hga_gather_kv + hga_attend (identical "
                         "results)")
    ap.add_argument("--routed-out", action="store_true",
                    help="fused gather: also write the gathered rows to the routed buffers "
                         "(k_routed, v_routed; bit-identical outputs); by default they stay in "
                         "the attention's LDS tiles")
    ap.add_argument("--route-from-q", action="store_true",
                    help="decode: hga_route forms q_bar from the query rows and the block's "
                         "summaries follow it (default: hga_build_summaries_qbar first, then "
                         "hga_route_qbar)")
    ap.add_argument("--schedule", default="graph-overlapped",
                    choices=("serial", "overlapped", "graph-serial", "graph-overlapped"),
                    help="decode sequence: route, gather and attend each block on one stream "
                         "(serial), or block b+1's gather on a second stream while block b "
                         "attends (overlapped); graph-*: the step replayed as a HIP graph "
                         "(default graph-overlapped)")
    ap.add_argument("--no-cache", action="store_true",
                    help="decode sequence: gather every block's routed groups from host memory")
    ap.add_argument("--cache-slots", type=int, default=0,
                    help="decode sequence: warm-cache slots per (batch, KV head) "
                         "(default 8 x topk_groups)")
    ap.add_argument("--backward", action="store_true",
                    help="time the attention backward (hga_attend_backward) of the workload")
    ap.add_argument("--block-exact", action="store_true",
                    help="with --blockwise: the single-workgroup attention whose outputs are "
                         "bit-identical to the bulk prefill's (default: the split attention)")
    ap.add_argument("--blockwise", action="store_true",
                    help="time the block-sequential prefill (hga_prefill_blocks) instead")
    ap.add_argument("--probe-traffic", action="store_true",
                    help="run attention and a known-size copy for rocprofv3 --pmc, then exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the library has no multi-GPU path (asked for "
              f"--gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_30709_amd import hga
    from paper_2606_30709_amd import workloads as W
    from paper_2606_30709_amd.pipeline import PrefillPipeline

    w = W.preset(args.workload)
    torch.cuda.set_device(0)
    inp = W.generate(w)
    if w.decode_block and w.decode_blocks > 1:
        decode_sequence_bench(w, inp, args)
        return
    if w.decode_block:
        decode_bench(w, inp, args)
        return
    if args.blockwise:
        blockwise_bench(w, inp, args)
        return
    if args.backward:
        backward_bench(w, inp, args)
        return
    if args.probe_traffic:
        probe_traffic(w, inp, args.gather, args.routed_out)
        return
    pipe = PrefillPipeline(w, inp, route_mode=args.route, gather_mode=args.gather,
                           routed_out=args.routed_out)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    p = pipe.plan

    summarise = lambda: hga.hga_build_summaries(p, pipe.k, 0, w.n_chunks, pipe.chunk_sum,
                                                pipe.group_sum, stream=sh)
    gather = lambda: hga.hga_gather_kv(p, pipe.group_idx, 0, pipe.k, pipe.v, pipe.k_routed,
                                       pipe.v_routed, stream=sh)
    if args.gather == "fused":
        # the dominant kernel's own dispatch records e0/e1 when given
        # with --routed-out the gathered rows are also written to the routed
        # buffers; by default they stay in the attention's LDS tiles
        kr, vr = (pipe.k_routed, pipe.v_routed) if args.routed_out else (None, None)
        attend_timed = lambda e0, e1: hga.hga_gather_attend(
            p, pipe.q, 0, pipe.k, pipe.v, pipe.group_idx, kr, vr, pipe.out, pipe.lse,
            start_event=e0, stop_event=e1, stream=sh)
        tail = (lambda: attend_timed(None, None),)
    else:
        attend_timed = lambda e0, e1: hga.hga_attend_timed(
            p, pipe.q, 0, pipe.k, pipe.v, pipe.k_routed, pipe.v_routed, pipe.group_idx, pipe.out,
            e0, e1, lse=pipe.lse, stream=sh)
        tail = (gather, lambda: hga.hga_attend(p, pipe.q, 0, pipe.k, pipe.v, pipe.k_routed,
                                               pipe.v_routed, pipe.group_idx, pipe.out,
                                               pipe.lse, stream=sh))
    stage_names = ROUTE_STAGES[args.route] + GATHER_STAGES[args.gather]
    att_name = stage_names[-1]
    if args.route == "separate":
        calls = (
            summarise,
            lambda: hga.hga_route_chunks(p, pipe.q, 0, pipe.chunk_sum, pipe.qbar, pipe.chunk_idx,
                                         stream=sh),
            lambda: hga.hga_route_groups(p, pipe.qbar, pipe.chunk_idx, 0, pipe.group_sum,
                                         pipe.group_idx, stream=sh)) + tail
    elif args.route == "fused":
        calls = (
            summarise,
            lambda: hga.hga_route(p, pipe.q, 0, pipe.chunk_sum, pipe.group_sum, pipe.qbar,
                                  pipe.chunk_idx, pipe.group_idx, stream=sh)) + tail
    else:
        calls = (
            lambda: hga.hga_build_summaries_qbar(p, pipe.k, 0, 0, w.n_chunks, pipe.chunk_sum,
                                                 pipe.group_sum, pipe.q, 0, pipe.qbar, stream=sh),
            lambda: hga.hga_route_qbar(p, pipe.qbar, 0, pipe.chunk_sum, pipe.group_sum,
                                       pipe.chunk_idx, pipe.group_idx, stream=sh)) + tail

    def one_step():
        for f in calls:
            f()

    settle(one_step, args.settle_seconds)
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    # Timed region: K steps; in a sample of them spread evenly over the
    # region (every `stride`-th step, at least ten, all of them for K <= 10)
    # the dominant kernel (attention) records a pair of HIP events at its own
    # dispatch start and end.  Recording events costs a few microseconds of
    # dispatch per step, so timing every step would lower the rate measured
    # for the whole region; whole-step rate from the wall clock between two
    # synchronizations.
    K = args.steps
    att = len(calls) - 1
    stride = max(1, K // 10)
    timed_steps = set(range(0, K, stride))
    ev_a = {s: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for s in timed_steps}
    for a, b in ev_a.values():  # events exist once recorded; the dispatch re-records them
        a.record(stream)
        b.record(stream)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for s in range(K):
        for n, f in enumerate(calls):
            if n == att and s in timed_steps:
                attend_timed(ev_a[s][0], ev_a[s][1])
            else:
                f()
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    attend_ms = float(np.mean([a.elapsed_time(b) for a, b in ev_a.values()]))
    gpu_step_ms = ev0.elapsed_time(ev1) / K

    # Breakdown pass (same workload, right after): events between all calls.
    KB = max(10, K // 2)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(KB)]
    torch.cuda.synchronize()
    for s in range(KB):
        ev[s][0].record(stream)
        for n, f in enumerate(calls):
            f()
            ev[s][n + 1].record(stream)
    torch.cuda.synchronize()
    stage_samples = {name: [ev[s][n].elapsed_time(ev[s][n + 1]) for s in range(KB)]
                     for n, name in enumerate(stage_names)}
    stage_samples[att_name] = [a.elapsed_time(b) for a, b in ev_a.values()]
    stage_ms = {name: float(np.mean(x)) for name, x in stage_samples.items()}
    stage_ms[att_name] = attend_ms
    wall_ms = (t1 - t0) * 1e3 / K
    tokens = w.batch * w.seq_len
    gi = pipe.group_idx.cpu().numpy()
    n_valid_rows = int((gi >= 0).sum()) * w.group
    abytes = algorithmic_bytes(w, n_valid_rows, pipe.routed_out)
    flops = attention_flops(w, gi)

    # achievable HBM bandwidth on this device, measured by a plain copy
    copy_gbs = measured_copy_bandwidth()
    dominant = max(stage_names, key=lambda s: stage_ms[s])
    stages = {}
    for sname in stage_names:
        sec = stage_ms[sname] * 1e-3
        p10, p50, p90 = np.percentile(stage_samples[sname], [10, 50, 90]) * 1e3
        ent = {"us": round(stage_ms[sname] * 1e3, 2),
               "p10_p50_p90_us": [round(float(p10), 2), round(float(p50), 2), round(float(p90), 2)],
               "alg_bytes": abytes[sname], "GB_s": round(abytes[sname] / sec / 1e9, 1),
               "hbm_frac": round(abytes[sname] / sec / 1e9 / HBM_PEAK_GBS, 4),
               "hbm_frac_of_copy": round(abytes[sname] / sec / 1e9 / copy_gbs, 4)}
        if sname in ATTENTION_STAGES:
            ent["TFLOP_s"] = round(flops / sec / 1e12, 2)
            ent["mfma_frac"] = round(flops / sec / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
        stages[sname] = ent
    dsec = stage_ms[dominant] * 1e-3
    # Bound by arithmetic intensity: attention above the ridge point (peak
    # compute / peak HBM bandwidth) is priced against the compute peak of its
    # own arithmetic (bf16 matrix cores, or fp32 vector ALUs for the fp32
    # kernel), everything else against HBM.
    cpeak, cbound = ((MFMA_BF16_PEAK_TFLOPS, "mfma") if w.dtype == "bf16"
                     else (VALU_FP32_PEAK_TFLOPS, "alu"))
    compute_bound = (dominant in ATTENTION_STAGES and
                     flops / abytes[dominant] > cpeak * 1e12 / (HBM_PEAK_GBS * 1e9))
    if compute_bound:
        achieved = flops / dsec / 1e12
        roofline = {"bound": cbound, "kernel": dominant, "achieved": round(achieved, 2),
                    "peak": cpeak, "unit": "TFLOP/s", "frac": round(achieved / cpeak, 4),
                    "alg_flops_per_launch": flops}
    else:
        achieved = abytes[dominant] / dsec / 1e9
        roofline = {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "copy_measured_GB_s": round(copy_gbs, 1),
                    "frac_of_copy": round(achieved / copy_gbs, 4)}
    roofline.update({
                "traffic": (measured_traffic(dominant, w.key, pipe.routed_out)
                            if dominant in ATTENTION_STAGES else None),
                "alg_bytes_per_launch": abytes[dominant],
                "mean_launch_us": round(stage_ms[dominant] * 1e3, 2),
                "timed_launches": len(timed_steps) if dominant == att_name else KB})

    res = {
        "metric": "routed-attn tokens/s per layer",
        "value": round(tokens * K / (t1 - t0), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{w.key}: prefill " + _prefill_label(w),
            "batch": w.batch, "seq_len": w.seq_len, "tokens_per_step": tokens,
            "seed": inp["seed"],
        },
        "gpu_ms_per_step_events": round(gpu_step_ms, 4),
        "stage_timing": (f"{att_name}: HIP events recorded by its own dispatch in "
                         f"{len(timed_steps)} of the {K} timed steps (every {stride}th); other "
                         "stages: a second pass of the same steps with events between all "
                         "calls"),
        "stages": stages,
        "route_calls": args.route,
        "gather_calls": args.gather,
        "routed_kv": ("written to the routed buffers" if pipe.routed_out else
                      "gathered into the attention's LDS tiles only (not written)"),
        "roofline": roofline,
        "device": torch.cuda.get_device_properties(0).gcnArchName,
    }
    if args.dense or w.key == "train12k":
        dense = dense_comparator(w, pipe)
        if dense.get("available"):
            dense["routed_speedup"] = round(res["value"] / dense["tokens_per_s"], 3)
        res["dense_comparator"] = dense
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
