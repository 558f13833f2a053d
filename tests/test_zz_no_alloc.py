"""hga_attend_split_static (the split attention with the library's static
per-device scratch instead of a caller workspace) against hga_attend_split
with a workspace of the same size: out and lse bit for bit, on two calls in a
row (the second with a smaller input), and the limit refused before any
launch.  Called through the C ABI."""

from __future__ import annotations

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_30709_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def hga():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_30709_amd import hga as H
    H.library()
    return H


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _decode_case():
    """A decode block: 64 queries of 32 heads over 4 KV heads (d128) after an
    8192-token history, compact resident hot chunks, routed buffers from the
    block's own routing."""
    from paper_2606_30709_amd.pipeline import DecodePipeline
    w = W.preset("decode64k").with_(seq_len=8192 + 64, needle_depths=(12, 64, 115))
    pipe = DecodePipeline(w, W.generate(w))
    pipe.route()
    pipe.gather()
    torch.cuda.synchronize()
    return dict(plan=pipe.plan, q=pipe.q, q_chunk0=pipe.c, k=pipe.k_res, v=pipe.v_res,
                kr=pipe.k_routed, vr=pipe.v_routed, gi=pipe.group_idx, res_slot=pipe.res_slot,
                label=f"decode block N{w.seq_len}")


def _prefill_case(key, **kw):
    """Query chunks [c0, c0 + n) of a prefill (token-indexed resident K/V)."""
    from paper_2606_30709_amd.pipeline import PrefillPipeline
    w = W.preset(key).with_(**kw)
    pipe = PrefillPipeline(w, W.generate(w))
    pipe.step()
    torch.cuda.synchronize()
    c0, n = w.n_chunks - 3, 3
    C = w.chunk
    return dict(plan=pipe.plan, q=pipe.q[:, :, c0 * C:(c0 + n) * C].contiguous(), q_chunk0=c0,
                k=pipe.k, v=pipe.v, kr=pipe.k_routed[:, :, c0:c0 + n].contiguous(),
                vr=pipe.v_routed[:, :, c0:c0 + n].contiguous(),
                gi=pipe.group_idx[:, :, c0:c0 + n].contiguous(), res_slot=None,
                label=f"{key} query chunks {c0}..{c0 + n - 1}")


def _both_ways(hga, case):
    """Outputs of the static entry point and of hga_attend_split with a
    workspace of the static array's size (NaN-poisoned outputs)."""
    nbytes = hga.hga_static_scratch_bytes()
    ws = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    outs = []
    for static in (True, False):
        out = torch.full_like(case["q"], float("nan"))
        lse = torch.full(case["q"].shape[:3], float("nan"), device="cuda")
        if static:
            hga.hga_attend_split_static(case["plan"], case["q"], case["q_chunk0"], case["k"],
                                        case["v"], case["kr"], case["vr"], case["gi"], out,
                                        lse=lse, res_slot=case["res_slot"])
        else:
            hga.hga_attend_split(case["plan"], case["q"], case["q_chunk0"], case["k"], case["v"],
                                 case["kr"], case["vr"], case["gi"], out, ws, lse=lse,
                                 res_slot=case["res_slot"])
        torch.cuda.synchronize()
        outs.append((out, lse))
    return outs


def test_static_scratch_split_attention_matches_workspace_form(hga):
    assert hga.hga_static_scratch_bytes() == 16 << 20
    first = _prefill_case("qwen32k", seq_len=4096)
    second = _decode_case()
    lib = hga.library()
    per = [lib.hga_attend_split_workspace(c["plan"].handle, c["q"].shape[2] // 64) // 16
           for c in (first, second)]
    assert per[1] < per[0], "the second call must be the smaller input"
    for case in (first, second):
        _say(f"[static scratch] {case['label']}")
        (o_s, l_s), (o_w, l_w) = _both_ways(hga, case)
        assert not torch.isnan(o_s).any() and not torch.isnan(l_s).any()
        assert torch.equal(_bits(o_s), _bits(o_w)), case["label"]
        assert torch.equal(l_s, l_w), case["label"]


def test_static_scratch_refuses_calls_beyond_its_size(hga):
    """Two splits of 32 query chunks of 32/4 heads at d128 need
    2 * 4 * 32 * 512 * 130 * 4 bytes = 68 MB, above the 16 MiB array: refused
    before any launch, outputs untouched."""
    case = _prefill_case("qwen32k", seq_len=4096)
    plan = case["plan"]
    C = 64
    n = 32
    q = torch.zeros(1, 32, n * C, 128, dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(q, 7.0)
    kr = torch.zeros(1, 4, n, plan.params.topk_groups * plan.params.group, 128,
                     dtype=torch.bfloat16, device="cuda")
    gi = torch.full((1, 4, n, plan.params.topk_groups), -1, dtype=torch.int32, device="cuda")
    with pytest.raises(hga.HgaError) as e:
        hga.hga_attend_split_static(plan, q, 0, case["k"], case["v"], kr, kr, gi, out)
    assert e.value.status == -2 and "static" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # a call within the limit still works afterwards, bit for bit as before
    second = _decode_case()
    (o_s, l_s), (o_w, l_w) = _both_ways(hga, second)
    assert torch.equal(_bits(o_s), _bits(o_w)) and torch.equal(l_s, l_w)
    assert np.isfinite(l_s.cpu().numpy()).all()
