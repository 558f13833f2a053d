"""The C-ABI library loads, exports every function include/hga.h declares,
and rejects bad parameters on the host (no GPU needed)."""

import ctypes
import os
import re

import pytest

from paper_2606_30709_amd import hga

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "hga.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hga_[a-z_]+)\s*\(", src)))


def test_header_declares_the_five_calls():
    names = _declared_functions()
    for n in ("hga_build_summaries", "hga_route_chunks", "hga_route_groups", "hga_route",
              "hga_gather_kv", "hga_attend"):
        assert n in names
    assert set(names) == set(hga.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(hga.library_path())
    for n in _declared_functions():
        assert hasattr(lib, n), n


def test_library_exports_nothing_undeclared():
    """Every hga_ function in the library's dynamic symbol table is declared
    in the header (no undocumented entry points)."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--defined-only", hga.library_path()], capture_output=True,
                         text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines()
                if len(l.split()) == 3 and l.split()[1] == "T" and l.split()[-1].startswith("hga_")}
    assert exported == set(_declared_functions())


def test_status_strings_and_version():
    for st in (0, -1, -2, -3, -4):
        assert hga.hga_status_string(st).startswith("HGA_")
    assert "unknown" in hga.hga_status_string(-99)
    assert hga.hga_version() >> 16 == 1


def _params(**kw):
    base = dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64, chunk=64, group=16,
                keep_first=1, keep_last=0, force_prev=1, topk_chunks=3, topk_groups=4,
                hf_pairs_chunk=-1, hf_pairs_group=-1, dtype=1, rope_base=1e4)
    base.update(kw)
    return hga.HgaParams(**base)


@pytest.mark.parametrize("bad,status", [
    (dict(n_q_heads=6, n_kv_heads=4), -1),
    (dict(head_dim=96), -2),
    (dict(chunk=128), -2),
    (dict(group=64), -2),
    (dict(group=12), -2),
    (dict(topk_chunks=0), -1),
    (dict(topk_groups=513), -1),
    (dict(keep_first=-1), -1),
    (dict(force_prev=2), -1),
    (dict(hf_pairs_chunk=33), -1),
    (dict(dtype=5), -1),
    (dict(rope_base=1.0), -1),
    (dict(rope_base=float("inf")), -1),
    (dict(batch=0), -1),
    (dict(hf_pairs_chunk=2, hf_pairs_group=5), -2),
    (dict(n_q_heads=34, n_kv_heads=2), -2),      # GQA ratio 17: above the tested 16
])
def test_plan_rejects_bad_params_before_touching_a_device(bad, status):
    lib = hga.library()
    p = _params(**bad)
    h = ctypes.c_void_p()
    assert lib.hga_plan_create(ctypes.byref(p), ctypes.byref(h)) == status
    assert h.value is None
    assert hga.hga_last_error()


def test_calls_reject_null_plan():
    lib = hga.library()
    assert lib.hga_build_summaries(None, None, 0, 0, 0, 0, None, None, 0, None) == -1
    assert lib.hga_route_chunks(None, None, 0, 0, None, 0, None, None, None) == -1
    assert lib.hga_route_groups(None, None, None, 0, 0, None, 0, None, None) == -1
    assert lib.hga_route(None, None, 0, 0, None, None, 0, None, None, None, None) == -1
    assert lib.hga_build_summaries_qbar(None, None, 0, 0, 0, 0, None, None, 0, None, 0, 0, None,
                                        None) == -1
    assert lib.hga_route_qbar(None, None, 0, 0, None, None, 0, None, None, None) == -1
    assert lib.hga_gather_kv(None, None, 0, 0, None, None, 0, 0, None, None, None) == -1
    assert lib.hga_attend(None, None, 0, 0, None, None, 0, None, None, None, None, None, None,
                          None) == -1
    assert lib.hga_attend_timed(None, None, 0, 0, None, None, 0, None, None, None, None, None,
                                None, None, None, None) == -1
    assert lib.hga_attend_split(None, None, 0, 0, None, None, 0, None, None, None, None, None,
                                None, None, 0, None) == -1
    assert lib.hga_attend_split_workspace(None, 1) == -1
    assert lib.hga_attend_split_static(None, None, 0, 0, None, None, 0, None, None, None, None,
                                       None, None, None) == -1
    assert lib.hga_static_scratch_bytes() == 16 << 20
    assert lib.hga_gather_attend_split(None, None, 0, 0, None, None, 0, None, None, None, 0, 0,
                                       None, None, None, None, None, None, 0, None) == -1
    assert lib.hga_gather_kv_cached(None, None, 0, None, None, 0, 0, None, None, 0, None, None,
                                    None, 0, None, 0, None, None, None, None) == -1
    assert lib.hga_attend_backward(None, None, 0, 0, None, None, 0, None, None, None, None, None,
                                   None, None, None) == -1
    assert lib.hga_gather_attend(None, None, 0, 0, None, None, 0, None, None, None, None, None,
                                 None, None, None) == -1
    assert lib.hga_block_step(None, None, 0, None, None, 0, None, None, 0, None, None, None,
                              None, None, None, None, None, 0, None) == -1
    assert lib.hga_prefill_blocks(None, None, 0, None, None, 0, None, None, 0, None, None, None,
                                  None, None, None, None, None, 0, None) == -1
    assert lib.hga_plan_destroy(None) == 0


def test_valid_plan_without_device_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    lib = hga.library()
    p = _params()
    h = ctypes.c_void_p()
    assert lib.hga_plan_create(ctypes.byref(p), ctypes.byref(h)) == -4
    assert h.value is None


@pytest.mark.parametrize("keep_first,keep_last,force_prev", [
    (1, 0, 1), (1, 0, 0), (2, 8, 1), (0, 3, 0), (4, 2, 1), (0, 0, 0), (3, 1, 0)])
def test_visible_chunks_follow_the_oracle(keep_first, keep_last, force_prev):
    """hga_visible_chunks (the enumeration the attention kernels use, host
    only) lists exactly the oracle's deterministic visible chunks D_c
    (Sec. 3.3) for every query chunk, and honours its capacity."""
    from oracle import hga_oracle as O
    p = _params(keep_first=keep_first, keep_last=keep_last, force_prev=force_prev)
    lib = hga.library()
    for c in range(0, 40):
        D, _ = O.visibility(c, keep_first, keep_last, force_prev)
        assert hga.hga_visible_chunks(p, c) == D, c
        if D:
            buf = (ctypes.c_int32 * 1)(-7)
            assert lib.hga_visible_chunks(ctypes.byref(p), c, ctypes.cast(buf, ctypes.c_void_p),
                                          1) == len(D)
            assert buf[0] == D[0]


def test_visible_chunks_reject_bad_input():
    lib = hga.library()
    p = _params()
    assert lib.hga_visible_chunks(ctypes.byref(p), -1, None, 0) == -1
    assert lib.hga_visible_chunks(ctypes.byref(p), 5, None, 3) == -1   # cap without a buffer
    bad = _params(head_dim=96)
    assert lib.hga_visible_chunks(ctypes.byref(bad), 5, None, 0) == -2
    assert lib.hga_visible_chunks(None, 5, None, 0) == -1
