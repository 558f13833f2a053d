"""GPU parity of the HIP path against the float64 oracle, called through the
C ABI (ctypes binding).  Every stage is compared on the GPU's own upstream
results (stage isolation): selections bit-exact with lowest-index ties unless
two candidates are within the fp32 error bound of each other; gathers
bit-exact; summaries and query means within their fp32 error bounds; outputs
within max-abs 1e-5 (fp32) / 2e-2 (bf16)."""

from __future__ import annotations

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import hga_oracle as O  # noqa: E402
from paper_2606_30709_amd import workloads as W  # noqa: E402

from parity_util import (BWD_TOL, LSE_TOL, OUT_TOL, SelectionReport, check_selection, f64,  # noqa: E402
                         score_bounds, summary_bound, tensor_to_f64)

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def hga():
    _need_gpu()
    from paper_2606_30709_amd import hga as H
    H.library()
    return H


# ------------------------------------------------------------ workloads ---

def W_(key, **kw):
    return W.preset(key).with_(**kw)


SMALL = {
    "tiny": W_("tiny"),
    "smalllm_2k": W_("smalllm", batch=2, seq_len=2048),
    "train_3k": W_("train12k", batch=2, n_q_heads=4, n_kv_heads=4, seq_len=3072),
    "qwen_4k": W_("qwen32k", seq_len=4096),
    "qwen_4k_ragged": W_("qwen32k", seq_len=4096, topk_groups=45, keep_last=3),
    "qwen_g8": W_("qwen32k", seq_len=2048, n_q_heads=8, n_kv_heads=2, group=8, topk_chunks=6,
                  topk_groups=21),
    "qwen_g32": W_("qwen32k", seq_len=2048, n_q_heads=8, n_kv_heads=2, group=32, topk_chunks=6,
                   topk_groups=7),
    "mha_d128": W_("qwen32k", seq_len=2048, n_q_heads=4, n_kv_heads=4, topk_chunks=5,
                   topk_groups=9),
    "gqa3_d64": W_("smalllm", batch=1, seq_len=2048, n_q_heads=6, n_kv_heads=2, topk_chunks=4,
                   topk_groups=7, keep_first=2, keep_last=1),
    # two query heads per KV head: the backward's fused form with four
    # wavefronts (d64) and its split form with a four-wavefront dQ (d128)
    "gqa2_d64": W_("smalllm", batch=1, seq_len=2048, n_q_heads=4, n_kv_heads=2, topk_chunks=4,
                   topk_groups=6),
    "gqa2_d128": W_("qwen32k", seq_len=2048, n_q_heads=4, n_kv_heads=2, topk_chunks=5,
                    topk_groups=9, keep_last=1),
    # four and sixteen query heads per KV head (the largest ratio the ABI accepts)
    "gqa4_d64": W_("smalllm", batch=1, seq_len=2048, n_q_heads=8, n_kv_heads=2, topk_chunks=4,
                   topk_groups=7),
    "gqa4_d128": W_("qwen32k", seq_len=2048, n_q_heads=8, n_kv_heads=2, topk_chunks=5,
                    topk_groups=9),
    "gqa16_d64": W_("smalllm", batch=1, seq_len=2048, n_q_heads=16, n_kv_heads=1, topk_chunks=4,
                    topk_groups=7),
    "gqa16_d128": W_("qwen32k", seq_len=2048, n_q_heads=32, n_kv_heads=2, topk_chunks=5,
                     topk_groups=9),
    "f32_gqa16": W_("tiny", n_q_heads=16, n_kv_heads=1),
    "tiny_noforce": W_("tiny", force_prev=0),
    "f32_d128_gqa": W_("tiny", seq_len=1024, n_q_heads=4, n_kv_heads=2, head_dim=128,
                       rope_base=1e6, topk_chunks=3, topk_groups=5, keep_last=2),
    # the chunk-only variant: every group of the routed chunks opened
    "qwen_chunks_4k": W_("qwen32k_chunks", seq_len=4096),
}


def _oracle_stage_checks(w, inp, pipe, units=None, chunk_ids=None):
    """Compare every stage of a finished PrefillPipeline with the oracle."""
    C, G, d = w.chunk, w.group, w.head_dim
    r = w.gqa_ratio
    q, k, v = (f64(inp[x], w.dtype) for x in "qkv")
    nc = w.n_chunks
    ids = list(range(nc)) if chunk_ids is None else chunk_ids
    nhc = O.high_freq_pairs(C, d, w.rope_base)
    nhg = O.high_freq_pairs(G, d, w.rope_base)
    assert pipe.plan.params.hf_pairs_chunk == nhc and pipe.plan.params.hf_pairs_group == nhg

    # summaries
    cs = O.summaries(k, C, w.rope_base, nhc)
    gs = O.summaries(k, G, w.rope_base, nhg)
    cmag = O.summary_magnitudes(k, C, w.rope_base, nhc)
    gmag = O.summary_magnitudes(k, G, w.rope_base, nhg)
    g_cs = tensor_to_f64(pipe.chunk_sum)
    g_gs = tensor_to_f64(pipe.group_sum)
    assert np.all(np.abs(g_cs - cs) <= summary_bound(cmag, C) + 1e-30), \
        f"chunk summaries: max err {np.max(np.abs(g_cs - cs)):.3g}"
    assert np.all(np.abs(g_gs - gs) <= summary_bound(gmag, G) + 1e-30), \
        f"group summaries: max err {np.max(np.abs(g_gs - gs)):.3g}"

    # query means
    qb = O.query_means(q, w.n_kv_heads, C)
    qmag = O.query_magnitudes(q, w.n_kv_heads, C)
    g_qb = tensor_to_f64(pipe.qbar)
    assert np.all(np.abs(g_qb - qb) <= 2 * (r * C + 8) * 2.0 ** -24 * qmag + 1e-30), \
        f"qbar: max err {np.max(np.abs(g_qb - qb)):.3g}"

    # chunk routing (oracle on exact inputs; near-tie rule)
    g_ci = pipe.chunk_idx.cpu().numpy()
    rep_c = SelectionReport()
    for c in ids:
        _, M = O.visibility(c, w.keep_first, w.keep_last, w.force_prev)
        for b in range(w.batch):
            for j in range(w.n_kv_heads):
                if not M:
                    assert np.all(g_ci[b, j, c] == -1)
                    continue
                sc = cs[b, j, M] @ qb[b, j, c]
                eps = score_bounds(qb[b, j, c], cs[b, j, M], qmag[b, j, c], cmag[b, j, M],
                                   C, r * C, d)
                check_selection(g_ci[b, j, c], M, sc, eps, w.topk_chunks, rep_c,
                                f"chunk_idx[{b},{j},{c}]")
    # group routing on the GPU's chunk selection
    g_gi = pipe.group_idx.cpu().numpy()
    rep_g = SelectionReport()
    gpc = C // G
    for c in ids:
        for b in range(w.batch):
            for j in range(w.n_kv_heads):
                chunks = [int(x) for x in g_ci[b, j, c] if x >= 0]
                if not chunks:
                    assert np.all(g_gi[b, j, c] == -1)
                    continue
                cand = np.array([cc * gpc + t for cc in chunks for t in range(gpc)])
                sc = gs[b, j, cand] @ qb[b, j, c]
                eps = score_bounds(qb[b, j, c], gs[b, j, cand], qmag[b, j, c], gmag[b, j, cand],
                                   G, r * C, d)
                check_selection(g_gi[b, j, c], cand, sc, eps, w.topk_groups, rep_g,
                                f"group_idx[{b},{j},{c}]")
    _say(f"  {w.key}: chunk selections {rep_c}, group selections {rep_g}")

    # gather: bit-exact on the GPU's group selection (when the step kept the
    # routed rows on chip, the standalone gather writes them for the check)
    if not pipe.routed_out:
        pipe.gather()
        torch.cuda.synchronize()
    kb = inp["k"]
    vb = inp["v"]
    sel = [(b, j, c) for b in range(w.batch) for j in range(w.n_kv_heads) for c in ids]
    gk = pipe.k_routed.cpu()
    gv = pipe.v_routed.cpu()
    if w.dtype == "bf16":
        gk, gv = gk.view(torch.int16).numpy().view(np.uint16), gv.view(torch.int16).numpy().view(np.uint16)
    else:
        gk, gv = gk.numpy(), gv.numpy()
    for (b, j, c) in sel:
        for s, g in enumerate(g_gi[b, j, c]):
            rows_k = gk[b, j, c, s * G:(s + 1) * G]
            rows_v = gv[b, j, c, s * G:(s + 1) * G]
            if g < 0:
                assert not np.any(rows_k) and not np.any(rows_v)
            else:
                assert np.array_equal(rows_k, kb[b, j, g * G:(g + 1) * G])
                assert np.array_equal(rows_v, vb[b, j, g * G:(g + 1) * G])

    # attention on the GPU's group selection
    if units is None:
        units = [(b, j, c) for b in range(w.batch) for j in range(w.n_kv_heads) for c in ids]
    out, lse = O.attend(q, k, v, g_gi, list(range(nc)), C, G, w.keep_first, w.keep_last,
                        w.force_prev, units=units)
    g_out = tensor_to_f64(pipe.out)
    g_lse = tensor_to_f64(pipe.lse)
    worst_o = worst_l = 0.0
    for (b, j, c) in units:
        hs = slice(j * r, (j + 1) * r)
        ts = slice(c * C, (c + 1) * C)
        eo = np.max(np.abs(g_out[b, hs, ts] - out[b, hs, ts]))
        el = np.max(np.abs(g_lse[b, hs, ts] - lse[b, hs, ts]))
        worst_o, worst_l = max(worst_o, eo), max(worst_l, el)
    _say(f"  {w.key}: out max-abs {worst_o:.3g} (tol {OUT_TOL[w.dtype]}), "
         f"lse max-abs {worst_l:.3g} (tol {LSE_TOL[w.dtype]})")
    assert worst_o <= OUT_TOL[w.dtype]
    assert worst_l <= LSE_TOL[w.dtype]
    return rep_c, rep_g


@pytest.mark.parametrize("key", list(SMALL))
def test_prefill_parity_small(hga, key):
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SMALL[key]
    _say(f"[parity] {key}: B{w.batch} H{w.n_q_heads}/{w.n_kv_heads} d{w.head_dim} N{w.seq_len} "
         f"{w.dtype} G{w.group} Kc{w.topk_chunks} Kg{w.topk_groups} F{w.keep_first} L{w.keep_last}")
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp)
    for t in (pipe.out, pipe.lse, pipe.chunk_sum, pipe.group_sum, pipe.qbar):
        t.fill_(float("nan"))
    pipe.chunk_idx.fill_(-7)
    pipe.group_idx.fill_(-7)
    pipe.step()
    torch.cuda.synchronize()
    assert not torch.isnan(pipe.out).any() and not torch.isnan(pipe.lse).any()
    _oracle_stage_checks(w, inp, pipe)


def test_planted_needles_routed_on_gpu(hga):
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SMALL["smalllm_2k"]
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp)
    pipe.step()
    ci = pipe.chunk_idx.cpu().numpy()
    for b, kc, qc in inp["needles"]:
        assert all(kc in ci[b, j, qc] for j in range(w.n_kv_heads))


def test_determinism_bitwise(hga):
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SMALL["qwen_4k"]
    pipe = PrefillPipeline(w, W.generate(w))
    pipe.step()
    first = [t.clone() for t in (pipe.chunk_sum, pipe.group_sum, pipe.qbar, pipe.chunk_idx,
                                 pipe.group_idx, pipe.k_routed, pipe.v_routed, pipe.out, pipe.lse)]
    pipe.step()
    second = (pipe.chunk_sum, pipe.group_sum, pipe.qbar, pipe.chunk_idx, pipe.group_idx,
              pipe.k_routed, pipe.v_routed, pipe.out, pipe.lse)
    for a, b in zip(first, second):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.uint8) if b.dtype == torch.bfloat16 else b)


# ---------------------------------------------------------- fused routing ---

def _route_both_ways(hga, plan, q, q_chunk0, cs, gs, nq, w):
    """Run hga_route_chunks + hga_route_groups and hga_route on the same inputs."""
    B, Hkv, d = w.batch, w.n_kv_heads, w.head_dim
    outs = []
    for fused in (False, True):
        qbar = torch.full((B, Hkv, nq, d), float("nan"), device="cuda")
        ci = torch.full((B, Hkv, nq, w.topk_chunks), -7, dtype=torch.int32, device="cuda")
        gi = torch.full((B, Hkv, nq, w.topk_groups), -7, dtype=torch.int32, device="cuda")
        if fused:
            hga.hga_route(plan, q, q_chunk0, cs, gs, qbar, ci, gi)
        else:
            hga.hga_route_chunks(plan, q, q_chunk0, cs, qbar, ci)
            hga.hga_route_groups(plan, qbar, ci, q_chunk0, gs, gi)
        outs.append((qbar, ci, gi))
    torch.cuda.synchronize()
    (qa, ca, ga), (qf, cf, gf) = outs
    assert torch.equal(qa.view(torch.int32), qf.view(torch.int32))
    assert torch.equal(ca, cf)
    assert torch.equal(ga, gf)
    assert (ca != -7).all() and (ga != -7).all()
    return ca, ga


FUSED_CASES = dict(SMALL, odd_37=W_("smalllm", batch=1, seq_len=37 * 64, topk_chunks=5,
                                    topk_groups=11))


@pytest.mark.parametrize("key", list(FUSED_CASES))
def test_fused_route_equals_separate_calls(hga, key):
    """hga_route writes exactly what hga_route_chunks + hga_route_groups write,
    for the whole sequence and for a query block starting mid-sequence."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = FUSED_CASES[key]
    _say(f"[fused-route] {key}")
    pipe = PrefillPipeline(w, W.generate(w))
    pipe.summaries()
    ca_all, ga_all = _route_both_ways(hga, pipe.plan, pipe.q, 0, pipe.chunk_sum,
                                      pipe.group_sum, w.n_chunks, w)
    # a ragged query block [c0, c0 + 5) of the same sequence routes as it did
    # inside the whole sequence
    c0 = w.n_chunks // 2 + 1
    n = min(5, w.n_chunks - c0)
    qb = pipe.q[:, :, c0 * w.chunk:(c0 + n) * w.chunk].contiguous()
    ca, ga = _route_both_ways(hga, pipe.plan, qb, c0, pipe.chunk_sum, pipe.group_sum, n, w)
    assert torch.equal(ca, ca_all[:, :, c0:c0 + n])
    assert torch.equal(ga, ga_all[:, :, c0:c0 + n])


# ------------------------------------------------- fused gather + attention ---

def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _gather_attend_both_ways(hga, plan, w, q, q_chunk0, k, v, gi):
    """hga_gather_kv + hga_attend and hga_gather_attend on the same inputs,
    every output pre-filled with NaN so that an unwritten element shows; and
    hga_gather_attend without routed buffers (rows gathered on chip only),
    whose out and lse must be the same bits."""
    B, Hkv, d, G = w.batch, w.n_kv_heads, w.head_dim, w.group
    nq = gi.shape[2]
    outs = []
    for mode in ("separate", "fused", "fused_no_routed"):
        kr = torch.full((B, Hkv, nq, w.topk_groups * G, d), float("nan"), dtype=k.dtype,
                        device="cuda")
        vr = torch.full_like(kr, float("nan"))
        out = torch.full_like(q, float("nan"))
        lse = torch.full(q.shape[:3], float("nan"), device="cuda")
        if mode == "fused":
            hga.hga_gather_attend(plan, q, q_chunk0, k, v, gi, kr, vr, out, lse)
        elif mode == "fused_no_routed":
            hga.hga_gather_attend(plan, q, q_chunk0, k, v, gi, None, None, out, lse)
        else:
            hga.hga_gather_kv(plan, gi, q_chunk0, k, v, kr, vr)
            hga.hga_attend(plan, q, q_chunk0, k, v, kr, vr, gi, out, lse)
        outs.append((kr, vr, out, lse))
    torch.cuda.synchronize()
    for a, b, name in zip(outs[0], outs[1], ("k_routed", "v_routed", "out", "lse")):
        assert torch.equal(_bits(a), _bits(b)), name
    assert not torch.isnan(outs[1][2]).any()
    for a, b, name in zip(outs[1][2:], outs[2][2:], ("out", "lse")):
        assert torch.equal(_bits(a), _bits(b)), f"{name} without routed buffers"
    # nothing was written to the routed buffers of the third call
    assert torch.isnan(outs[2][0]).all() and torch.isnan(outs[2][1]).all()


@pytest.mark.parametrize("key", list(FUSED_CASES))
def test_gather_attend_equals_separate_calls(hga, key):
    """hga_gather_attend writes exactly what hga_gather_kv + hga_attend write:
    the routed buffers, the output and the LSE, bit for bit; for the whole
    sequence, with padded and out-of-range group ids planted, and for a query
    block starting mid-sequence."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = FUSED_CASES[key]
    _say(f"[gather-attend] {key}")
    pipe = PrefillPipeline(w, W.generate(w), gather_mode="separate")
    pipe.summaries()
    pipe.route()
    _gather_attend_both_ways(hga, pipe.plan, w, pipe.q, 0, pipe.k, pipe.v, pipe.group_idx)
    gi = pipe.group_idx.clone()
    c = w.n_chunks - 1
    gi[0, 0, c, 0] = -1
    gi[0, w.n_kv_heads - 1, c, w.topk_groups - 1] = 10 ** 6  # beyond the causal past
    gi[-1, 0, c // 2, w.topk_groups // 2] = -1
    _gather_attend_both_ways(hga, pipe.plan, w, pipe.q, 0, pipe.k, pipe.v, gi)
    c0 = w.n_chunks // 3
    n = min(5, w.n_chunks - c0)
    C = w.chunk
    q_blk = pipe.q[:, :, c0 * C:(c0 + n) * C].contiguous()
    gi_blk = pipe.group_idx[:, :, c0:c0 + n].contiguous()
    _gather_attend_both_ways(hga, pipe.plan, w, q_blk, c0, pipe.k, pipe.v, gi_blk)


SPLIT_CASES = {k: SMALL[k] for k in ("qwen_4k_ragged", "qwen_g8", "qwen_g32", "gqa3_d64",
                                     "mha_d128", "f32_d128_gqa", "gqa4_d64", "gqa16_d64",
                                     "gqa4_d128", "gqa16_d128")}


BWD_CASES = {k: SMALL[k] for k in ("smalllm_2k", "gqa2_d64", "gqa2_d128", "gqa3_d64",
                                   "gqa4_d64", "gqa4_d128", "gqa16_d64", "gqa16_d128",
                                   "qwen_4k_ragged", "qwen_g8",
                                   "qwen_g32", "mha_d128", "qwen_chunks_4k")}


@pytest.mark.parametrize("key", list(BWD_CASES))
def test_attend_backward_matches_oracle(hga, key):
    """hga_attend_backward against the oracle's chain rule (float64, on the
    GPU's routing and with a seeded output gradient): dq, dk, dv within the
    bar derived from the bf16 rounding of the weights and of dS."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = BWD_CASES[key]
    _say(f"[backward] {key}")
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp)
    pipe.step()
    rng = np.random.default_rng(77)
    dout_f = rng.standard_normal(pipe.q.shape).astype(np.float32)
    dout = torch.from_numpy(dout_f).to(torch.bfloat16).cuda()
    dq, dk, dv = pipe.backward(dout)
    torch.cuda.synchronize()
    q64, k64, v64 = (f64(inp[x], w.dtype) for x in "qkv")
    go = dout.float().cpu().numpy().astype(np.float64)
    rq, rk, rv = O.attend_backward(
        q64, k64, v64, go, pipe.group_idx.cpu().numpy(), list(range(w.n_chunks)), w.chunk,
        w.group, w.keep_first, w.keep_last, w.force_prev)
    for name, g, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        g = g.cpu().numpy().astype(np.float64)
        assert np.isfinite(g).all(), name
        err = np.max(np.abs(g - ref))
        scale = np.max(np.abs(ref))
        rel = np.linalg.norm(g - ref) / np.linalg.norm(ref)
        _say(f"  {name}: max-abs {err:.3g} of max {scale:.3g} ({err / scale:.3g}), "
             f"normwise {rel:.3g}")
        assert err <= BWD_TOL * scale and rel <= BWD_TOL / 4, name


@pytest.mark.parametrize("key", ["smalllm_2k", "gqa3_d64", "qwen_4k_ragged"])
def test_attend_backward_query_block_offset(hga, key):
    """hga_attend_backward on the last two query chunks alone (q_chunk0 > 0,
    as for a block's gradient): dq of those rows, and dk, dv holding only
    their contributions, against the oracle on the same chunk ids; both
    backward forms (fused for smalllm_2k, split for the GQA cases)."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SMALL[key]
    _say(f"[backward-offset] {key}")
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp)
    pipe.step()
    C, q0 = w.chunk, w.n_chunks - 2
    rows = slice(q0 * C, w.n_chunks * C)
    q = pipe.q[:, :, rows].contiguous()
    out = pipe.out[:, :, rows].contiguous()
    lse = pipe.lse[:, :, rows].contiguous()
    gi = pipe.group_idx[:, :, q0:].contiguous()
    rng = np.random.default_rng(78)
    dout = torch.from_numpy(rng.standard_normal(q.shape).astype(np.float32)).to(torch.bfloat16).cuda()
    dq = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    dk = torch.zeros(pipe.k.shape, dtype=torch.float32, device="cuda")
    dv = torch.zeros_like(dk)
    hga.hga_attend_backward(pipe.plan, q, q0, pipe.k, pipe.v, gi, out, lse, dout, dq, dk, dv)
    torch.cuda.synchronize()
    q64, k64, v64 = (f64(inp[x], w.dtype) for x in "qkv")
    rq, rk, rv = O.attend_backward(
        q64[:, :, rows], k64, v64, dout.float().cpu().numpy().astype(np.float64),
        gi.cpu().numpy(), [q0, q0 + 1], C, w.group, w.keep_first, w.keep_last, w.force_prev)
    for name, g, ref in (("dq", dq, rq), ("dk", dk, rk), ("dv", dv, rv)):
        g = g.cpu().numpy().astype(np.float64)
        assert np.isfinite(g).all(), name
        err = np.max(np.abs(g - ref))
        scale = np.max(np.abs(ref))
        rel = np.linalg.norm(g - ref) / np.linalg.norm(ref)
        _say(f"  {name}: max-abs {err:.3g} of max {scale:.3g}, normwise {rel:.3g}")
        assert err <= BWD_TOL * scale and rel <= BWD_TOL / 4, name


@pytest.mark.parametrize("key", list(SPLIT_CASES))
def test_attend_split_matches_oracle(hga, key):
    """hga_attend_split computes the same softmax as hga_attend with its
    partial sums (and the bf16 rounding of its weights, taken against each
    split's own reference point) in another order: its outputs meet the
    oracle bar on single query chunks (the first ones have padded routing, so
    some splits see only masked rows), on a multi-chunk block and with planted
    invalid group ids; where it runs as one split (fp32, one head per KV
    head, a workspace too small for two, none) it is hga_attend bit for bit."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SPLIT_CASES[key]
    _say(f"[attend-split] {key}")
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp, gather_mode="separate")
    pipe.step()
    plan, C, r = pipe.plan, w.chunk, w.gqa_ratio
    q64, k64, v64 = (f64(inp[x], w.dtype) for x in "qkv")
    nbytes = hga.hga_attend_split_workspace(plan, 3)
    ws = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")

    def run(c0, n, gi, split, workspace=ws):
        q = pipe.q[:, :, c0 * C:(c0 + n) * C].contiguous()
        kr = pipe.k_routed[:, :, c0:c0 + n].contiguous()
        vr = pipe.v_routed[:, :, c0:c0 + n].contiguous()
        out = torch.full_like(q, float("nan"))
        lse = torch.full(q.shape[:3], float("nan"), device="cuda")
        if split:
            hga.hga_attend_split(plan, q, c0, pipe.k, pipe.v, kr, vr, gi, out, workspace, lse)
        else:
            hga.hga_attend(plan, q, c0, pipe.k, pipe.v, kr, vr, gi, out, lse)
        torch.cuda.synchronize()
        return out, lse

    def check(c0, n, gi_np):
        gi = torch.from_numpy(np.ascontiguousarray(gi_np[:, :, c0:c0 + n])).cuda()
        out, lse = run(c0, n, gi, True)
        units = [(b, j, c) for b in range(w.batch) for j in range(w.n_kv_heads)
                 for c in range(c0, c0 + n)]
        # the calls treat an id outside [0, c * C / G) as an absent slot (the
        # routing never produces one); the oracle is given -1 there
        lim = (np.arange(w.n_chunks) * (C // w.group))[None, None, :, None]
        gi_ref = np.where((gi_np >= 0) & (gi_np < lim), gi_np, -1)
        o_ref, l_ref = O.attend(q64, k64, v64, gi_ref, list(range(w.n_chunks)), C, w.group,
                                w.keep_first, w.keep_last, w.force_prev, units=units)
        ts = slice(c0 * C, (c0 + n) * C)
        eo = np.max(np.abs(tensor_to_f64(out) - o_ref[:, :, ts]))
        el = np.max(np.abs(tensor_to_f64(lse) - l_ref[:, :, ts]))
        po, pl = run(c0, n, gi, False)
        gap = float((po.float() - out.float()).abs().max())
        _say(f"  chunks {c0}..{c0 + n - 1}: out {eo:.3g} lse {el:.3g} (vs hga_attend {gap:.3g})")
        assert eo <= OUT_TOL[w.dtype] and el <= LSE_TOL[w.dtype]
        return out, lse, po, pl

    gi_np = pipe.group_idx.cpu().numpy()
    for c in sorted({0, 1, 2, 3, w.n_chunks // 2, w.n_chunks - 1}):
        out, lse, po, pl = check(c, 1, gi_np)
        if not (w.dtype == "bf16" and r >= 2):
            assert torch.equal(_bits(out), _bits(po)) and torch.equal(lse, pl)
    check(w.n_chunks // 3, 3, gi_np)
    planted = gi_np.copy()
    c = w.n_chunks - 1
    planted[0, 0, c, 0] = -1
    planted[0, w.n_kv_heads - 1, c, w.topk_groups - 1] = 10 ** 6
    check(c, 1, planted)
    # a workspace below two splits' worth (one split of one chunk is
    # nbytes / 48 bytes), or none: hga_attend itself
    gi = pipe.group_idx[:, :, c:c + 1].contiguous()
    po, pl = run(c, 1, gi, False)
    for small in (ws[: nbytes // 96 - 1], None):
        out, lse = run(c, 1, gi, True, workspace=small)
        assert torch.equal(_bits(out), _bits(po)) and torch.equal(lse, pl)


@pytest.mark.parametrize("key", ["qwen_4k_ragged", "gqa3_d64", "f32_d128_gqa", "mha_d128"])
def test_gather_attend_split_without_routed_buffers(hga, key):
    """hga_gather_attend_split from device-resident sources, on prefill-layout
    query blocks: the routed rows it writes are hga_gather_kv's, and with
    both routed buffers NULL (rows gathered on chip only) its output and LSE
    are the same bits, also with padded and out-of-range group ids."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SPLIT_CASES[key]
    _say(f"[gather-attend-split, no routed buffers] {key}")
    pipe = PrefillPipeline(w, W.generate(w), gather_mode="separate")
    pipe.summaries()
    pipe.route()
    pipe.gather()
    torch.cuda.synchronize()
    C = w.chunk
    planted = pipe.group_idx.clone()
    c = w.n_chunks - 1
    planted[0, 0, c, 0] = -1
    planted[0, w.n_kv_heads - 1, c, w.topk_groups - 1] = 10 ** 6
    for gi_all, c0, n in ((pipe.group_idx, 0, 1), (pipe.group_idx, w.n_chunks // 3, 3),
                          (planted, c, 1)):
        q = pipe.q[:, :, c0 * C:(c0 + n) * C].contiguous()
        gi = gi_all[:, :, c0:c0 + n].contiguous()
        ws = torch.empty(hga.hga_attend_split_workspace(pipe.plan, n) // 4,
                         dtype=torch.float32, device="cuda")
        kr = torch.full_like(pipe.k_routed[:, :, c0:c0 + n], float("nan"))
        vr = torch.full_like(kr, float("nan"))
        outs = []
        for routed in ((kr, vr), (None, None)):
            out = torch.full_like(q, float("nan"))
            lse = torch.full(q.shape[:3], float("nan"), device="cuda")
            hga.hga_gather_attend_split(pipe.plan, q, c0, pipe.k, pipe.v, pipe.k, pipe.v, gi,
                                        routed[0], routed[1], out, ws, lse)
            torch.cuda.synchronize()
            outs.append((out, lse))
        if gi_all is pipe.group_idx:  # the separate gather ran on these ids
            assert torch.equal(_bits(kr), _bits(pipe.k_routed[:, :, c0:c0 + n]))
            assert torch.equal(_bits(vr), _bits(pipe.v_routed[:, :, c0:c0 + n]))
        (o1, l1), (o2, l2) = outs
        assert not torch.isnan(o1).any() and not torch.isnan(l1).any()
        assert torch.equal(_bits(o1), _bits(o2)) and torch.equal(l1, l2)


def test_gather_attend_full_size(hga):
    """The fused call equals the two calls at the full prefill sizes."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    for key in ("smalllm", "train12k", "qwen32k"):
        w = W.preset(key)
        _say(f"[gather-attend] {key} full size")
        pipe = PrefillPipeline(w, W.generate(w), gather_mode="separate")
        pipe.summaries()
        pipe.route()
        _gather_attend_both_ways(hga, pipe.plan, w, pipe.q, 0, pipe.k, pipe.v, pipe.group_idx)
        del pipe
        torch.cuda.empty_cache()


# ------------------------------------------------ block-sequential prefill ---

BLOCK_CASES = {k: SMALL[k] for k in ("tiny", "smalllm_2k", "qwen_4k_ragged", "qwen_g8",
                                      "gqa3_d64", "qwen_chunks_4k")}


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("key", list(BLOCK_CASES))
def test_block_sequential_prefill_equals_bulk(hga, key, split):
    """Prefill as a sequence of 64-token blocks (route against the chunks
    closed so far, attend, append) writes, block by block, exactly what the
    bulk prefill writes for the same query chunk: prefill = decode.  With the
    split attention (a workspace) the summaries, routing and routed buffers
    are still identical and the outputs meet the oracle bar."""
    from paper_2606_30709_amd.pipeline import BlockPrefillPipeline, PrefillPipeline
    w = BLOCK_CASES[key]
    _say(f"[block-prefill] {key} split={split}")
    inp = W.generate(w)
    bulk = PrefillPipeline(w, inp)
    bulk.step()
    blk = BlockPrefillPipeline(w, inp, split_attend=split)
    for t in (blk.out, blk.lse, blk.qbar):
        t.fill_(float("nan"))
    blk.chunk_idx.fill_(-7)
    blk.group_idx.fill_(-7)
    blk.step()
    torch.cuda.synchronize()
    nc, C = w.n_chunks, w.chunk
    B, Hq, d = w.batch, w.n_q_heads, w.head_dim
    same = lambda a, b: torch.equal(_bits(a.contiguous()), _bits(b.contiguous()))
    assert same(blk.chunk_sum, bulk.chunk_sum) and same(blk.group_sum, bulk.group_sum)
    # block-major -> bulk layouts
    assert same(blk.qbar[:, :, :, 0].permute(1, 2, 0, 3), bulk.qbar)
    assert torch.equal(blk.chunk_idx[:, :, :, 0].permute(1, 2, 0, 3), bulk.chunk_idx)
    assert torch.equal(blk.group_idx[:, :, :, 0].permute(1, 2, 0, 3), bulk.group_idx)
    assert same(blk.k_routed[:, :, :, 0].permute(1, 2, 0, 3, 4), bulk.k_routed)
    assert same(blk.v_routed[:, :, :, 0].permute(1, 2, 0, 3, 4), bulk.v_routed)
    out_bulk = bulk.out.reshape(B, Hq, nc, C, d).permute(2, 0, 1, 3, 4)
    lse_bulk = bulk.lse.reshape(B, Hq, nc, C).permute(2, 0, 1, 3)
    if not split:
        assert same(blk.out, out_bulk)
        assert same(blk.lse, lse_bulk)
        return
    assert not torch.isnan(blk.out).any() and not torch.isnan(blk.lse).any()
    chunks = sorted({0, 1, nc // 2, nc - 1})
    q64, k64, v64 = (f64(inp[x], w.dtype) for x in "qkv")
    units = [(b, j, c) for b in range(B) for j in range(w.n_kv_heads) for c in chunks]
    o_ref, l_ref = O.attend(q64, k64, v64, bulk.group_idx.cpu().numpy(), list(range(nc)), C,
                            w.group, w.keep_first, w.keep_last, w.force_prev, units=units)
    g_out = tensor_to_f64(blk.out)
    g_lse = tensor_to_f64(blk.lse)
    eo = max(np.max(np.abs(g_out[c] - o_ref[:, :, c * C:(c + 1) * C])) for c in chunks)
    el = max(np.max(np.abs(g_lse[c] - l_ref[:, :, c * C:(c + 1) * C])) for c in chunks)
    _say(f"  split blocks {chunks}: out {eo:.3g} lse {el:.3g}")
    assert eo <= OUT_TOL[w.dtype] and el <= LSE_TOL[w.dtype]


def _split_route_check(hga, plan, k, k_chunk0, n_chunks, table_chunks, q, q_chunk0, w):
    """hga_build_summaries_qbar + hga_route_qbar against hga_build_summaries +
    hga_route, bit for bit."""
    B, Hkv, d, C, G = w.batch, w.n_kv_heads, w.head_dim, w.chunk, w.group
    nq = q.shape[2] // C
    outs = []
    for split in (False, True):
        cs = torch.full((B, Hkv, table_chunks, d), float("nan"), device="cuda")
        gs = torch.full((B, Hkv, table_chunks * (C // G), d), float("nan"), device="cuda")
        qbar = torch.full((B, Hkv, nq, d), float("nan"), device="cuda")
        ci = torch.full((B, Hkv, nq, w.topk_chunks), -7, dtype=torch.int32, device="cuda")
        gi = torch.full((B, Hkv, nq, w.topk_groups), -7, dtype=torch.int32, device="cuda")
        if split:
            hga.hga_build_summaries_qbar(plan, k, k_chunk0, k_chunk0, k_chunk0 + n_chunks, cs, gs,
                                         q, q_chunk0, qbar)
            hga.hga_route_qbar(plan, qbar, q_chunk0, cs, gs, ci, gi)
        else:
            hga.hga_build_summaries(plan, k, k_chunk0, k_chunk0 + n_chunks, cs, gs)
            hga.hga_route(plan, q, q_chunk0, cs, gs, qbar, ci, gi)
        outs.append((cs, gs, qbar, ci, gi))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("key", list(FUSED_CASES))
def test_summaries_qbar_and_route_qbar_equal_fused(hga, key):
    """The summaries + query means launch and the routing from that q_bar
    write what the summaries call and hga_route write."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = FUSED_CASES[key]
    _say(f"[split-route] {key}")
    pipe = PrefillPipeline(w, W.generate(w))
    _split_route_check(hga, pipe.plan, pipe.k, 0, w.n_chunks, w.n_chunks, pipe.q, 0, w)
    # a query block mid-sequence, summaries of every chunk before its end
    c0 = w.n_chunks // 2 + 1
    n = min(5, w.n_chunks - c0)
    qb = pipe.q[:, :, c0 * w.chunk:(c0 + n) * w.chunk].contiguous()
    _split_route_check(hga, pipe.plan, pipe.k, 0, c0 + n, w.n_chunks, qb, c0, w)


def test_summaries_qbar_decode_and_full_size(hga):
    from paper_2606_30709_amd.pipeline import DecodePipeline, PrefillPipeline
    w = W.preset("decode64k")
    _say("[split-route] decode64k")
    pipe = DecodePipeline(w, W.generate(w))
    # the history's summaries from a device copy, then the block's routing
    k_dev = pipe.k_hist.to("cuda")
    _split_route_check(hga, pipe.plan, k_dev, 0, pipe.c, pipe.c + 1, pipe.q, pipe.c, w)
    del k_dev
    for key in ("smalllm", "qwen32k"):
        w = W.preset(key)
        _say(f"[split-route] {key}")
        pipe = PrefillPipeline(w, W.generate(w))
        _split_route_check(hga, pipe.plan, pipe.k, 0, w.n_chunks, w.n_chunks, pipe.q, 0, w)


def test_fused_route_decode_and_full_size(hga):
    from paper_2606_30709_amd.pipeline import DecodePipeline, PrefillPipeline
    w = W.preset("decode64k")
    _say("[fused-route] decode64k")
    pipe = DecodePipeline(w, W.generate(w))
    _route_both_ways(hga, pipe.plan, pipe.q, pipe.c, pipe.chunk_sum, pipe.group_sum, 1, w)
    for key in ("smalllm", "qwen32k"):
        w = W.preset(key)
        _say(f"[fused-route] {key}")
        pipe = PrefillPipeline(w, W.generate(w))
        pipe.summaries()
        _route_both_ways(hga, pipe.plan, pipe.q, 0, pipe.chunk_sum, pipe.group_sum,
                         w.n_chunks, w)


def test_attend_timed_records_kernel_events(hga):
    """hga_attend_timed writes what hga_attend writes, and its dispatch records
    the two events (a positive duration between them)."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    for key in ("smalllm_2k", "tiny"):
        w = SMALL[key]
        pipe = PrefillPipeline(w, W.generate(w))
        pipe.step()
        torch.cuda.synchronize()
        ref_o, ref_l = pipe.out.clone(), pipe.lse.clone()
        pipe.out.fill_(float("nan"))
        pipe.lse.fill_(float("nan"))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        e1.record()
        hga.hga_attend_timed(pipe.plan, pipe.q, 0, pipe.k, pipe.v, pipe.k_routed, pipe.v_routed,
                             pipe.group_idx, pipe.out, e0, e1, lse=pipe.lse)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        _say(f"[timed] {key}: {ms * 1e3:.1f} us")
        assert ms > 0
        assert torch.equal(pipe.out.view(torch.uint8), ref_o.view(torch.uint8))
        assert torch.equal(pipe.lse, ref_l)


# ----------------------------------------------------------------- decode ---

def _decode_check(hga, w):
    from paper_2606_30709_amd.pipeline import DecodePipeline
    inp = W.generate(w)
    pipe = DecodePipeline(w, inp)
    pipe.out.fill_(float("nan"))
    pipe.step()
    torch.cuda.synchronize()
    C, G, d, r = w.chunk, w.group, w.head_dim, w.gqa_ratio
    c = w.q_chunk0
    q, k, v = (f64(inp[x], w.dtype) for x in "qkv")
    nhc = O.high_freq_pairs(C, d, w.rope_base)
    nhg = O.high_freq_pairs(G, d, w.rope_base)
    cs = O.summaries(k, C, w.rope_base, nhc)
    gs = O.summaries(k, G, w.rope_base, nhg)
    cmag = O.summary_magnitudes(k, C, w.rope_base, nhc)
    gmag = O.summary_magnitudes(k, G, w.rope_base, nhg)
    qb = O.query_means(q, w.n_kv_heads, C)
    qmag = O.query_magnitudes(q, w.n_kv_heads, C)
    # summaries of the history and of the appended block
    g_cs = tensor_to_f64(pipe.chunk_sum)
    assert np.all(np.abs(g_cs - cs) <= summary_bound(cmag, C) + 1e-30)
    g_gs = tensor_to_f64(pipe.group_sum)
    assert np.all(np.abs(g_gs - gs) <= summary_bound(gmag, G) + 1e-30)
    _, M = O.visibility(c, w.keep_first, w.keep_last, w.force_prev)
    g_ci = pipe.chunk_idx.cpu().numpy()
    g_gi = pipe.group_idx.cpu().numpy()
    rc, rg = SelectionReport(), SelectionReport()
    gpc = C // G
    for b in range(w.batch):
        for j in range(w.n_kv_heads):
            sc = cs[b, j, M] @ qb[b, j, 0]
            eps = score_bounds(qb[b, j, 0], cs[b, j, M], qmag[b, j, 0], cmag[b, j, M], C, r * C, d)
            check_selection(g_ci[b, j, 0], M, sc, eps, w.topk_chunks, rc, f"decode chunk {b},{j}")
            chunks = [int(x) for x in g_ci[b, j, 0] if x >= 0]
            cand = np.array([cc * gpc + t for cc in chunks for t in range(gpc)])
            sc = gs[b, j, cand] @ qb[b, j, 0]
            eps = score_bounds(qb[b, j, 0], gs[b, j, cand], qmag[b, j, 0], gmag[b, j, cand],
                               G, r * C, d)
            check_selection(g_gi[b, j, 0], cand, sc, eps, w.topk_groups, rg, f"decode group {b},{j}")
    out, lse = O.attend(q, k, v, g_gi, [c], C, G, w.keep_first, w.keep_last, w.force_prev)
    eo = np.max(np.abs(tensor_to_f64(pipe.out) - out))
    el = np.max(np.abs(tensor_to_f64(pipe.lse) - lse))
    _say(f"  decode {w.key} N{w.seq_len}: {rc} {rg} out {eo:.3g} lse {el:.3g} "
         f"pcie bytes {pipe.pcie_bytes_per_step()}")
    assert eo <= OUT_TOL[w.dtype] and el <= LSE_TOL[w.dtype]
    # needles at the configured depths are routed for every KV head
    for kc, _ in inp["needles"]:
        if kc in M:
            assert all(kc in g_ci[0, j, 0] for j in range(w.n_kv_heads)), f"needle {kc} missed"
    return pipe


def test_decode_fused_gather_equals_separate(hga):
    """The host gather inside the split attention (hga_gather_attend_split)
    writes exactly what hga_gather_kv from host memory + hga_attend_split
    write: routed buffers, output and LSE, bit for bit; also with padded and
    future group ids planted."""
    from paper_2606_30709_amd.pipeline import DecodePipeline
    for w in (W.preset("decode64k"), W_("decode64k", seq_len=8192 + 64,
                                        needle_depths=(12, 64, 115))):
        _say(f"[decode fused gather] N{w.seq_len}")
        inp = W.generate(w)
        fused = DecodePipeline(w, inp, fused_gather=True)
        sep = DecodePipeline(w, inp, plan=fused.plan)
        assert fused.fused_gather and not sep.fused_gather
        for pipe in (fused, sep):
            pipe.route()
        torch.cuda.synchronize()
        assert torch.equal(fused.group_idx, sep.group_idx)
        for planted in (False, True):
            if planted:
                for pipe in (fused, sep):
                    pipe.group_idx[0, 0, 0, 0] = -1
                    pipe.group_idx[0, w.n_kv_heads - 1, 0, w.topk_groups - 1] = 10 ** 6
            for pipe in (fused, sep):
                for t in (pipe.k_routed, pipe.v_routed, pipe.out, pipe.lse):
                    t.fill_(float("nan"))
            fused.gather_attend()
            sep.gather()
            sep.attend()
            torch.cuda.synchronize()
            for name in ("k_routed", "v_routed", "out", "lse"):
                a, b = getattr(fused, name), getattr(sep, name)
                assert torch.equal(_bits(a), _bits(b)), name
            assert not torch.isnan(fused.out).any()
            # without routed buffers: the same output and LSE bits
            out2 = torch.full_like(fused.out, float("nan"))
            lse2 = torch.full_like(fused.lse, float("nan"))
            hga.hga_gather_attend_split(fused.plan, fused.q, fused.c, fused.k_res, fused.v_res,
                                        fused.k_hist, fused.v_hist, fused.group_idx, None, None,
                                        out2, fused.attend_ws, lse2, res_slot=fused.res_slot,
                                        src_on_host=True)
            torch.cuda.synchronize()
            assert torch.equal(_bits(out2), _bits(fused.out))
            assert torch.equal(lse2, fused.lse)


class _LruModel:
    """The warm cache's replacement rule in plain Python: per (batch, KV
    head), hits keep their slot; misses take the slots not used in this call
    with the oldest last use (never-used first, then the lowest slot), in
    ascending slot order, in routed order; a repeated id is served once."""

    def __init__(self, n_units, n_slots):
        self.n_slots = n_slots
        self.sg = [[-1] * n_slots for _ in range(n_units)]
        self.su = [[-1] * n_slots for _ in range(n_units)]
        self.gs = [dict() for _ in range(n_units)]

    def call(self, unit, ids, lim, tick):
        sg, su, gs = self.sg[unit], self.su[unit], self.gs[unit]
        seen, hits, misses = set(), set(), []
        for g in ids:
            if not (0 <= g < lim) or g in seen:
                continue
            seen.add(g)
            v = gs.get(g, -1)
            if v >= 0 and sg[v] == g:
                hits.add(v)
            else:
                misses.append(g)
        for v in hits:
            su[v] = tick
        cand = sorted((su[v], v) for v in range(self.n_slots) if v not in hits)
        victims = sorted(v for _, v in cand[:len(misses)])
        for g, v in zip(misses, victims):
            old = sg[v]
            if old >= 0 and gs.get(old) == v:
                del gs[old]
            sg[v], gs[g], su[v] = g, v, tick
        return len(misses)


@pytest.mark.parametrize("slots_per_topk", [1, 4])
def test_warm_cache_gather(hga, slots_per_topk):
    """Consecutive decode blocks through the warm LRU cache of routed groups:
    every block's routed buffers and outputs equal those of the uncached host
    gather bit for bit, the per-head count of groups fetched from host memory
    and the final slot maps follow the LRU model, every occupied slot holds
    its group's rows, and the last block meets the oracle bar.  Run twice
    over the sequence (the second pass starts warm)."""
    from paper_2606_30709_amd.pipeline import DecodeSequencePipeline
    w = W_("decode64k_seq", seq_len=8192 + 16 * 64, needle_depths=(12, 64, 115))
    n_slots = slots_per_topk * w.topk_groups
    _say(f"[warm cache] {n_slots} slots, {w.decode_blocks} blocks")
    inp = W.generate(w)
    cached = DecodeSequencePipeline(w, inp, cache_slots=n_slots)
    plain = DecodeSequencePipeline(w, inp, plan=cached.plan)
    B, Hkv, C, G = w.batch, w.n_kv_heads, w.chunk, w.group
    model = _LruModel(B * Hkv, n_slots)
    src_tokens = cached.k_hist.shape[2]
    fetched_total = 0
    for rep in range(2):
        for b in range(w.decode_blocks):
            tick = cached.cache.tick
            cached.block(b)
            plain.block(b)
            torch.cuda.synchronize()
            assert torch.equal(cached.group_idx[b], plain.group_idx[b])
            for name in ("k_routed", "v_routed"):
                assert torch.equal(_bits(getattr(cached, name)), _bits(getattr(plain, name))), name
            assert torch.equal(_bits(cached.out[b]), _bits(plain.out[b]))
            assert torch.equal(cached.lse[b], plain.lse[b])
            c = cached.c0 + b
            lim = min(c * (C // G), src_tokens // G)
            gi = cached.group_idx[b].cpu().numpy()
            got = cached.n_fetched[b].cpu().numpy()
            for bb in range(B):
                for j in range(Hkv):
                    exp = model.call(bb * Hkv + j, [int(x) for x in gi[bb, j, 0]], lim, tick)
                    assert got[bb, j] == exp, (rep, b, bb, j, got[bb, j], exp)
                    fetched_total += exp
        _say(f"  pass {rep}: {int(cached.n_fetched.sum())} of "
             f"{int((cached.group_idx >= 0).sum())} routed groups fetched from host")
    sg = cached.cache.slot_group.cpu().numpy().reshape(B * Hkv, n_slots)
    assert sg.tolist() == model.sg
    kh = cached.k_hist
    ck = cached.cache.k.cpu()
    for bb in range(B):
        for j in range(Hkv):
            for v in range(n_slots):
                g = int(sg[bb * Hkv + j, v])
                if g >= 0:
                    assert torch.equal(_bits(ck[bb, j, v]), _bits(kh[bb, j, g * G:(g + 1) * G]))
    # the last block against the oracle
    b = w.decode_blocks - 1
    c = cached.c0 + b
    q64, k64, v64 = (f64(inp[x], w.dtype) for x in "qkv")
    gi_all = cached.group_idx[:, :, :, 0].permute(1, 2, 0, 3).cpu().numpy()   # [B, Hkv, nb, K]
    units = [(bb, j, b) for bb in range(B) for j in range(Hkv)]
    o_ref, l_ref = O.attend(q64, k64, v64, gi_all, list(range(cached.c0, cached.c0 + w.decode_blocks)),
                            C, G, w.keep_first, w.keep_last, w.force_prev, units=units)
    eo = np.max(np.abs(tensor_to_f64(cached.out[b]) - o_ref[:, :, b * C:(b + 1) * C]))
    el = np.max(np.abs(tensor_to_f64(cached.lse[b]) - l_ref[:, :, b * C:(b + 1) * C]))
    _say(f"  block {c}: out {eo:.3g} lse {el:.3g}")
    assert eo <= OUT_TOL[w.dtype] and el <= LSE_TOL[w.dtype]
    # planted repeats and invalid ids in one call
    gi = cached.group_idx[b].clone()
    gi[0, 0, 0, 1] = gi[0, 0, 0, 0]
    gi[0, 1, 0, 2] = -1
    gi[0, 2, 0, 3] = 10 ** 6
    kr, vr = torch.empty_like(cached.k_routed), torch.empty_like(cached.v_routed)
    tick = cached.cache.tick
    hga.hga_gather_kv_cached(cached.plan, gi, c, cached.k_hist, cached.v_hist, cached.cache,
                             kr, vr, cached.n_fetched[0], src_on_host=True)
    kp, vp = torch.empty_like(kr), torch.empty_like(vr)
    hga.hga_gather_kv(cached.plan, gi, c, cached.k_hist, cached.v_hist, kp, vp, src_on_host=True)
    torch.cuda.synchronize()
    assert torch.equal(_bits(kr), _bits(kp)) and torch.equal(_bits(vr), _bits(vp))
    got = cached.n_fetched[0].cpu().numpy()
    lim = min(c * (C // G), src_tokens // G)
    gnp = gi.cpu().numpy()
    for bb in range(B):
        for j in range(Hkv):
            assert got[bb, j] == model.call(bb * Hkv + j, [int(x) for x in gnp[bb, j, 0]], lim, tick)


def test_decode_sequence_overlapped_equals_serial(hga):
    """The two-stream decode schedule (block b+1's gather, through the warm
    cache or straight from host memory, on a second stream while block b
    attends) writes exactly what the one-stream schedule writes: every
    block's routing, output and LSE, the per-block miss counts, the final
    cache maps and the last block's routed buffers; run twice over the
    sequence (cold, then warm)."""
    from paper_2606_30709_amd.pipeline import DecodeSequencePipeline
    w = W_("decode64k_seq", seq_len=8192 + 16 * 64, needle_depths=(12, 64, 115))
    inp = W.generate(w)
    n_slots = 4 * w.topk_groups
    _say(f"[decode overlap] {w.decode_blocks} blocks, {n_slots} slots")
    serial = DecodeSequencePipeline(w, inp, cache_slots=n_slots)
    over = DecodeSequencePipeline(w, inp, plan=serial.plan, cache_slots=n_slots)
    plain = DecodeSequencePipeline(w, inp, plan=serial.plan)
    last = w.decode_blocks - 1
    for rep in range(2):
        for pipe in (serial, over, plain):
            pipe.out.fill_(float("nan"))
            pipe.lse.fill_(float("nan"))
            pipe.group_idx.fill_(-7)
        serial.step()
        over.step_overlapped()
        plain.step_overlapped()
        torch.cuda.synchronize()
        assert torch.equal(serial.group_idx, over.group_idx)
        assert torch.equal(serial.group_idx, plain.group_idx)
        for pipe in (over, plain):
            assert torch.equal(_bits(serial.out), _bits(pipe.out))
            assert torch.equal(serial.lse, pipe.lse)
        assert torch.equal(serial.n_fetched, over.n_fetched)
        assert torch.equal(_bits(serial.k_routed), _bits(over.k_routed2[last % 2]))
        assert torch.equal(_bits(serial.v_routed), _bits(plain.v_routed2[last % 2]))
        _say(f"  pass {rep}: {int(over.n_fetched.sum())} groups fetched from host")
    for name in ("slot_group", "slot_used", "group_slot"):
        assert torch.equal(getattr(serial.cache, name), getattr(over.cache, name)), name
    assert not torch.isnan(over.out).any()


@pytest.mark.parametrize("overlapped", [True, False])
def test_decode_sequence_graph_replays_equal_eager(hga, overlapped):
    """The decode sequence (16 blocks through the warm cache) recorded as a
    HIP graph: three replays, each after emptying the cache and with eager
    work of another pipeline in between, write exactly what one eager step
    from an empty cache writes (routing, outputs, LSE, miss counts, the
    cache's slot maps)."""
    from paper_2606_30709_amd.pipeline import DecodeSequencePipeline
    w = W_("decode64k_seq", seq_len=8192 + 16 * 64, needle_depths=(12, 64, 115))
    inp = W.generate(w)
    n_slots = 4 * w.topk_groups
    _say(f"[decode graph] overlapped={overlapped}")
    ref = DecodeSequencePipeline(w, inp, cache_slots=n_slots)
    ref.reset_cache()
    ref.step()
    torch.cuda.synchronize()
    want = {k: getattr(ref, k).clone() for k in ("out", "lse", "group_idx", "n_fetched")}
    want_maps = {k: getattr(ref.cache, k).clone() for k in ("slot_group", "group_slot")}
    pipe = DecodeSequencePipeline(w, inp, plan=ref.plan, cache_slots=n_slots)
    g = pipe.capture(overlapped)
    for rep in range(3):
        for name in ("out", "lse"):
            getattr(pipe, name).fill_(float("nan"))
        pipe.reset_cache()
        g.replay()
        ref.reset_cache()
        ref.step()                      # eager work between the replays
        torch.cuda.synchronize()
        assert torch.equal(_bits(pipe.out), _bits(want["out"])), rep
        assert torch.equal(pipe.lse, want["lse"]), rep
        assert torch.equal(pipe.group_idx, want["group_idx"]), rep
        assert torch.equal(pipe.n_fetched, want["n_fetched"]), rep
        for k, v in want_maps.items():
            assert torch.equal(getattr(pipe.cache, k), v), (rep, k)


def test_decode_block_parity_reduced(hga):
    w = W_("decode64k", seq_len=8192 + 64, needle_depths=(12, 64, 115))
    _decode_check(hga, w)


def test_decode_block_parity_128k(hga):
    """A context beyond 64K: 2037 routable chunks per unit (the wide route's
    selection with two candidates per thread), history of 131,072 tokens in
    pinned host memory."""
    _decode_check(hga, W.preset("decode128k"))


def test_decode_block_parity_128k_wrapped_positions(hga):
    """The same 128K context with RoPE positions taken modulo 65536 (Sec. 5,
    long-context positional encoding): the keys past 64K repeat the first
    positions' rotations; routing and attention are unchanged code and still
    match the oracle on these inputs."""
    _decode_check(hga, W_("decode128k", rope_wrap=65536))


def test_decode_block_parity_full(hga):
    pipe = _decode_check(hga, W.preset("decode64k"))
    # host-sourced gather equals a device-sourced gather of the same history
    kd, vd = pipe.k_hist.to("cuda"), pipe.v_hist.to("cuda")
    k2, v2 = torch.empty_like(pipe.k_routed), torch.empty_like(pipe.v_routed)
    hga.hga_gather_kv(pipe.plan, pipe.group_idx, pipe.c, kd, vd, k2, v2)
    torch.cuda.synchronize()
    assert torch.equal(k2.view(torch.int16), pipe.k_routed.view(torch.int16))
    assert torch.equal(v2.view(torch.int16), pipe.v_routed.view(torch.int16))


# -------------------------------------------------------------- full size ---

@pytest.mark.parametrize("key", ["smalllm", "train12k", "qwen32k", "qwen32k_chunks"])
def test_prefill_parity_full_size_sampled(hga, key):
    """Full sizes, launched exactly as the benchmark does; the oracle checks
    every summary and query mean, the routing of sampled query chunks, and
    the attention of every query chunk of one (batch, KV head) -- or, with
    four KV heads, of 64 units, each head's first and last chunks included."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = W.preset(key)
    _say(f"[full] {key}")
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp, routed_out=False)  # the benchmark's form
    pipe.out.fill_(float("nan"))
    pipe.step()
    torch.cuda.synchronize()
    assert not torch.isnan(pipe.out).any()
    rng = np.random.default_rng(5)
    nc = w.n_chunks
    chunk_ids = sorted(set([0, 1, 2, 3, nc - 1] + list(rng.choice(nc, 6, replace=False))))
    if w.n_kv_heads * w.batch > 4:
        # every query chunk of one (batch, KV head)
        b0, j0 = int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads))
        units = [(b0, j0, c) for c in range(nc)]
    else:
        # 64 units: the first and last chunks of every KV head, the rest drawn
        units = sorted(set([(b, j, c) for b in range(w.batch) for j in range(w.n_kv_heads)
                            for c in (0, 1, nc - 1)]))
        while len(units) < 64:
            u = (int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads)),
                 int(rng.integers(nc)))
            if u not in units:
                units.append(u)
    _say(f"  attention checked on {len(units)} units")
    _oracle_stage_checks(w, inp, pipe, units=units, chunk_ids=chunk_ids)


# ------------------------------------------------------------- edge cases ---

def test_argument_errors_launch_nothing(hga):
    w = SMALL["tiny"]
    plan = hga.Plan.for_workload(w)
    dev = "cuda"
    k = torch.zeros(1, 1, 1024, 64, device=dev)
    cs = torch.zeros(1, 1, 16, 64, device=dev)
    gs = torch.zeros(1, 1, 64, 64, device=dev)
    with pytest.raises(hga.HgaError) as e:
        hga.hga_build_summaries(plan, k, 0, 17, cs, gs)          # beyond table
    assert e.value.status == -1
    with pytest.raises(hga.HgaError):
        hga.hga_build_summaries(plan, k[:, :, :512], 0, 16, cs, gs)   # K too short
    lib = hga.library()
    st = lib.hga_build_summaries(plan.handle, k.data_ptr() + 4, 1024, 0, 0, 16, cs.data_ptr(),
                                 gs.data_ptr(), 16, None)
    assert st == -3                                              # misaligned
    st = lib.hga_route_chunks(plan.handle, None, 0, 16, cs.data_ptr(), 16, cs.data_ptr(),
                              cs.data_ptr(), None)
    assert st == -1
    q = torch.zeros(1, 1, 1024, 64, device=dev)
    st = lib.hga_route_chunks(plan.handle, q.data_ptr(), 5, 16, cs.data_ptr(), 16,
                              cs.data_ptr(), cs.data_ptr(), None)
    assert st == -1                                              # needs table of 20 chunks
    st = lib.hga_attend(plan.handle, q.data_ptr(), 0, 16, k.data_ptr(), k.data_ptr(), 512, None,
                        k.data_ptr(), k.data_ptr(), cs.data_ptr(), q.data_ptr(), None, None)
    assert st == -1                                              # resident K/V too short
    host = torch.zeros(1, 1, 1024, 64)                           # pageable host memory
    gi = torch.zeros(1, 1, 16, 4, dtype=torch.int32, device=dev)
    kr = torch.zeros(1, 1, 16, 64, 64, device=dev)
    st = lib.hga_gather_kv(plan.handle, gi.data_ptr(), 0, 16, host.data_ptr(), host.data_ptr(),
                           1024, 1, kr.data_ptr(), kr.data_ptr(), None)
    assert st == -1
    assert "pinned" in hga.hga_last_error()
    # the fused gather's source must cover the causal past of the last query chunk
    st = lib.hga_gather_attend_split(plan.handle, q.data_ptr(), 0, 16, k.data_ptr(),
                                     k.data_ptr(), 1024, None, k.data_ptr(), k.data_ptr(), 900, 0,
                                     gi.data_ptr(), kr.data_ptr(), kr.data_ptr(), q.data_ptr(),
                                     None, None, 0, None)
    assert st == -1 and "causal past" in hga.hga_last_error()
    st = lib.hga_gather_attend_split(plan.handle, q.data_ptr(), 0, 16, k.data_ptr(),
                                     k.data_ptr(), 1024, None, host.data_ptr(), host.data_ptr(),
                                     1024, 1, gi.data_ptr(), kr.data_ptr(), kr.data_ptr(),
                                     q.data_ptr(), None, None, 0, None)
    assert st == -1 and "pinned" in hga.hga_last_error()
    # the routed buffers of the fused gathers: both or neither
    kk = torch.zeros(1, 1, 1024, 64, device=dev)
    for kr_p, vr_p in ((kr.data_ptr(), None), (None, kr.data_ptr())):
        st = lib.hga_gather_attend(plan.handle, q.data_ptr(), 0, 16, kk.data_ptr(),
                                   kk.data_ptr(), 1024, gi.data_ptr(), kr_p, vr_p, q.data_ptr(),
                                   None, None, None, None)
        assert st == -1 and "both" in hga.hga_last_error()
        st = lib.hga_gather_attend_split(plan.handle, q.data_ptr(), 0, 16, kk.data_ptr(),
                                         kk.data_ptr(), 1024, None, kk.data_ptr(), kk.data_ptr(),
                                         1024, 0, gi.data_ptr(), kr_p, vr_p, q.data_ptr(), None,
                                         None, 0, None)
        assert st == -1 and "both" in hga.hga_last_error()
    # empty ranges are no-ops
    hga.hga_build_summaries(plan, k, 3, 3, cs, gs)
    torch.cuda.synchronize()


def test_backward_argument_errors(hga):
    """hga_attend_backward refuses, before any launch: an fp32 plan
    (unsupported), a missing lse, and resident K/V that do not cover the
    query chunks; the outputs stay untouched."""
    lib = hga.library()
    dev = "cuda"
    plan32 = hga.Plan.for_workload(SMALL["tiny"])
    q = torch.zeros(1, 1, 1024, 64, device=dev)
    k = torch.zeros(1, 1, 1024, 64, device=dev)
    gi = torch.zeros(1, 1, 16, 4, dtype=torch.int32, device=dev)
    lse = torch.zeros(1, 1, 1024, device=dev)
    st = lib.hga_attend_backward(plan32.handle, q.data_ptr(), 0, 16, k.data_ptr(), k.data_ptr(),
                                 1024, gi.data_ptr(), q.data_ptr(), lse.data_ptr(), q.data_ptr(),
                                 q.data_ptr(), q.data_ptr(), q.data_ptr(), None)
    assert st == -2 and "bf16" in hga.hga_last_error()
    w = SMALL["smalllm_2k"]
    plan = hga.Plan.for_workload(w)
    B, Hq, Hkv, d, N = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.seq_len
    qb = torch.zeros(B, Hq, N, d, dtype=torch.bfloat16, device=dev)
    kb = torch.zeros(B, Hkv, N, d, dtype=torch.bfloat16, device=dev)
    gib = torch.zeros(B, Hkv, w.n_chunks, w.topk_groups, dtype=torch.int32, device=dev)
    lseb = torch.zeros(B, Hq, N, device=dev)
    dq = torch.full((B, Hq, N, d), 7.0, device=dev)
    dk = torch.full((B, Hkv, N, d), 7.0, device=dev)
    args = lambda lse_ptr, res: (plan.handle, qb.data_ptr(), 0, w.n_chunks, kb.data_ptr(),
                                 kb.data_ptr(), res, gib.data_ptr(), qb.data_ptr(), lse_ptr,
                                 qb.data_ptr(), dq.data_ptr(), dk.data_ptr(), dk.data_ptr(), None)
    assert lib.hga_attend_backward(*args(None, N)) == -1
    assert "lse" in hga.hga_last_error()
    assert lib.hga_attend_backward(*args(lseb.data_ptr(), N - 64)) == -1
    torch.cuda.synchronize()
    assert bool((dq == 7.0).all()) and bool((dk == 7.0).all())


def test_gather_and_attend_handle_invalid_slots(hga):
    """-1 and out-of-range group ids give zero rows in the gather and are
    skipped by attention; an invalid resident slot poisons its rows."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = SMALL["qwen_g8"]
    inp = W.generate(w)
    pipe = PrefillPipeline(w, inp)
    pipe.step()
    gi = pipe.group_idx.clone()
    c = w.n_chunks - 1
    gi[0, 0, c, 3] = -1
    gi[0, 1, c, 5] = 10 ** 6         # beyond the causal past
    pipe.group_idx.copy_(gi)
    pipe.gather()
    pipe.attend()
    torch.cuda.synchronize()
    G = w.group
    assert not pipe.k_routed[0, 0, c, 3 * G:4 * G].any()
    assert not pipe.v_routed[0, 1, c, 5 * G:6 * G].any()
    q, k, v = (f64(inp[x], w.dtype) for x in "qkv")
    gnp = gi.cpu().numpy()
    # the C ABI ignores ids outside [0, c * chunk/group) like -1: tell the oracle so
    gpc = w.chunk // G
    for cc in range(w.n_chunks):
        sl = gnp[:, :, cc]
        sl[(sl < 0) | (sl >= cc * gpc)] = -1
    units = [(0, 0, c), (0, 1, c)]
    out, _ = O.attend(q, k, v, gnp, list(range(w.n_chunks)), w.chunk, G, w.keep_first,
                      w.keep_last, w.force_prev, units=units)
    g_out = tensor_to_f64(pipe.out)
    r = w.gqa_ratio
    for (b, j, cc) in units:
        sl = (b, slice(j * r, (j + 1) * r), slice(cc * 64, (cc + 1) * 64))
        assert np.max(np.abs(g_out[sl] - out[sl])) <= OUT_TOL[w.dtype]
    # resident-slot indirection: identity map equals no map; an invalid slot gives NaN rows
    slot = torch.arange(w.n_chunks, dtype=torch.int32, device="cuda")
    out2 = torch.empty_like(pipe.out)
    hga.hga_attend(pipe.plan, pipe.q, 0, pipe.k, pipe.v, pipe.k_routed, pipe.v_routed,
                   pipe.group_idx, out2, None, res_slot=slot)
    torch.cuda.synchronize()
    assert torch.equal(out2.view(torch.int16), pipe.out.view(torch.int16))
    slot[c] = 999
    hga.hga_attend(pipe.plan, pipe.q, 0, pipe.k, pipe.v, pipe.k_routed, pipe.v_routed,
                   pipe.group_idx, out2, None, res_slot=slot)
    torch.cuda.synchronize()
    assert torch.isnan(out2[:, :, c * 64:(c + 1) * 64]).all()
    assert not torch.isnan(out2[:, :, :c * 64]).any()


def test_incremental_summaries_equal_bulk(hga):
    """Appending chunk by chunk (the store's append) equals one bulk build."""
    w = SMALL["qwen_4k"]
    inp = W.generate(w)
    from paper_2606_30709_amd.pipeline import to_device
    k = to_device(inp["k"], w.dtype)
    plan = hga.Plan.for_workload(w)
    nc = w.n_chunks
    shape_c = (w.batch, w.n_kv_heads, nc, w.head_dim)
    shape_g = (w.batch, w.n_kv_heads, nc * 4, w.head_dim)
    a_c, a_g = torch.zeros(shape_c, device="cuda"), torch.zeros(shape_g, device="cuda")
    b_c, b_g = torch.zeros(shape_c, device="cuda"), torch.zeros(shape_g, device="cuda")
    hga.hga_build_summaries(plan, k, 0, nc, a_c, a_g)
    for c in range(nc):
        blk = k[:, :, c * 64:(c + 1) * 64].contiguous()
        hga.hga_build_summaries(plan, blk, c, c + 1, b_c, b_g, k_chunk0=c)
    torch.cuda.synchronize()
    assert torch.equal(a_c, b_c) and torch.equal(a_g, b_g)
