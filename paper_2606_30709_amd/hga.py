"""Thin ctypes binding of libhga.so (include/hga.h).

Argument marshalling only: tensors are passed as raw device pointers with the
sizes read from their shapes, and the stream is torch's current stream unless
one is given.  Every step of the routed-attention path runs in the library's
HIP kernels; there is no fallback.  If the library is missing, importing the
binding's functions raises.
"""

from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "HgaError", "HgaParams", "Plan", "WarmCache", "library", "library_path", "F32", "BF16",
    "hga_build_summaries", "hga_route_chunks", "hga_route_groups", "hga_route",
    "hga_build_summaries_qbar", "hga_route_qbar", "hga_gather_kv", "hga_attend",
    "hga_attend_timed", "hga_attend_split", "hga_attend_split_workspace",
    "hga_attend_split_static", "hga_static_scratch_bytes", "hga_gather_attend",
    "hga_gather_attend_split", "hga_gather_kv_cached", "hga_attend_backward",
    "hga_block_step", "hga_prefill_blocks", "hga_status_string", "hga_last_error",
    "hga_version", "hga_visible_chunks", "EXPORTED_SYMBOLS",
]

F32, BF16 = 0, 1
_TORCH_DTYPE = {F32: torch.float32, BF16: torch.bfloat16}

EXPORTED_SYMBOLS = (
    "hga_plan_create", "hga_plan_destroy", "hga_plan_params", "hga_build_summaries",
    "hga_route_chunks", "hga_route_groups", "hga_route", "hga_build_summaries_qbar",
    "hga_route_qbar", "hga_gather_kv", "hga_attend", "hga_attend_timed", "hga_attend_split",
    "hga_attend_split_workspace", "hga_attend_split_static", "hga_static_scratch_bytes",
    "hga_gather_attend", "hga_gather_attend_split",
    "hga_gather_kv_cached", "hga_attend_backward", "hga_block_step", "hga_prefill_blocks",
    "hga_status_string",
    "hga_last_error", "hga_version", "hga_visible_chunks",
)


class HgaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} [status {status}]")
        self.status = status


class HgaParams(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("chunk", ctypes.c_int32), ("group", ctypes.c_int32),
        ("keep_first", ctypes.c_int32), ("keep_last", ctypes.c_int32),
        ("force_prev", ctypes.c_int32), ("topk_chunks", ctypes.c_int32),
        ("topk_groups", ctypes.c_int32), ("hf_pairs_chunk", ctypes.c_int32),
        ("hf_pairs_group", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("rope_base", ctypes.c_double),
    ]


def library_path() -> str:
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhga.so")


_LIB = None


def library() -> ctypes.CDLL:
    """Load libhga.so (after torch, so both share torch's HIP runtime)."""
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            raise ImportError(f"{path} is not built; run `python -m paper_2606_30709_amd.build`")
        lib = ctypes.CDLL(path)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        sigs = {
            "hga_plan_create": [ctypes.POINTER(HgaParams), ctypes.POINTER(vp)],
            "hga_plan_destroy": [vp],
            "hga_plan_params": [vp, ctypes.POINTER(HgaParams)],
            "hga_build_summaries": [vp, vp, i64, i32, i32, i32, vp, vp, i32, vp],
            "hga_route_chunks": [vp, vp, i32, i32, vp, i32, vp, vp, vp],
            "hga_route_groups": [vp, vp, vp, i32, i32, vp, i32, vp, vp],
            "hga_route": [vp, vp, i32, i32, vp, vp, i32, vp, vp, vp, vp],
            "hga_build_summaries_qbar": [vp, vp, i64, i32, i32, i32, vp, vp, i32, vp, i32, i32,
                                         vp, vp],
            "hga_route_qbar": [vp, vp, i32, i32, vp, vp, i32, vp, vp, vp],
            "hga_gather_kv": [vp, vp, i32, i32, vp, vp, i64, i32, vp, vp, vp],
            "hga_gather_kv_cached": [vp, vp, i32, vp, vp, i64, i32, vp, vp, i32, vp, vp, vp, i64,
                                     vp, i32, vp, vp, vp, vp],
            "hga_attend": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp],
            "hga_attend_timed": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp],
            "hga_attend_split": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, i64,
                                 vp],
            "hga_attend_split_static": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp,
                                        vp],
            "hga_gather_attend": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp],
            "hga_attend_backward": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp,
                                    vp],
            "hga_gather_attend_split": [vp, vp, i32, i32, vp, vp, i64, vp, vp, vp, i64, i32, vp,
                                        vp, vp, vp, vp, vp, i64, vp],
            "hga_block_step": [vp, vp, i32, vp, vp, i64, vp, vp, i32, vp, vp, vp, vp, vp, vp,
                               vp, vp, i64, vp],
            "hga_prefill_blocks": [vp, vp, i32, vp, vp, i64, vp, vp, i32, vp, vp, vp, vp, vp,
                                   vp, vp, vp, i64, vp],
        }
        for name, args in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = i32
        lib.hga_attend_split_workspace.argtypes = [vp, i32]
        lib.hga_attend_split_workspace.restype = i64
        lib.hga_static_scratch_bytes.argtypes = []
        lib.hga_static_scratch_bytes.restype = i64
        lib.hga_status_string.argtypes = [i32]
        lib.hga_status_string.restype = ctypes.c_char_p
        lib.hga_last_error.argtypes = []
        lib.hga_last_error.restype = ctypes.c_char_p
        lib.hga_version.argtypes = []
        lib.hga_version.restype = i32
        lib.hga_visible_chunks.argtypes = [ctypes.POINTER(HgaParams), i32, vp, i32]
        lib.hga_visible_chunks.restype = i32
        _LIB = lib
    return _LIB


def hga_status_string(status: int) -> str:
    return library().hga_status_string(status).decode()


def hga_last_error() -> str:
    return library().hga_last_error().decode()


def hga_version() -> int:
    return library().hga_version()


def hga_visible_chunks(params: HgaParams, c: int) -> list:
    """The closed chunks query chunk c sees besides its own, ascending (the
    library's enumeration; host only)."""
    n = library().hga_visible_chunks(ctypes.byref(params), c, None, 0)
    if n < 0:
        raise HgaError(n, hga_last_error())
    buf = (ctypes.c_int32 * max(n, 1))()
    _check(min(0, library().hga_visible_chunks(ctypes.byref(params), c,
                                               ctypes.cast(buf, ctypes.c_void_p), n)))
    return list(buf[:n])


def _check(status: int):
    if status != 0:
        raise HgaError(status, f"{hga_status_string(status)}: {hga_last_error()}")


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Plan:
    """Owns an hga_plan (the resolved routing configuration and the summary
    phase tables on the current device)."""

    def __init__(self, *, batch, n_q_heads, n_kv_heads, head_dim, chunk=64, group=16,
                 keep_first=1, keep_last=0, force_prev=1, topk_chunks, topk_groups,
                 hf_pairs_chunk=-1, hf_pairs_group=-1, dtype=BF16, rope_base=10000.0):
        self._handle = None
        p = HgaParams(batch, n_q_heads, n_kv_heads, head_dim, chunk, group, keep_first,
                      keep_last, force_prev, topk_chunks, topk_groups, hf_pairs_chunk,
                      hf_pairs_group, dtype, float(rope_base))
        h = ctypes.c_void_p()
        _check(library().hga_plan_create(ctypes.byref(p), ctypes.byref(h)))
        self._handle = h
        out = HgaParams()
        _check(library().hga_plan_params(h, ctypes.byref(out)))
        self.params = out

    @classmethod
    def for_workload(cls, w, **overrides):
        kw = dict(batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                  head_dim=w.head_dim, chunk=w.chunk, group=w.group, keep_first=w.keep_first,
                  keep_last=w.keep_last, force_prev=w.force_prev, topk_chunks=w.topk_chunks,
                  topk_groups=w.topk_groups, dtype=F32 if w.dtype == "f32" else BF16,
                  rope_base=w.rope_base)
        kw.update(overrides)
        return cls(**kw)

    @property
    def handle(self):
        if self._handle is None:
            raise RuntimeError("plan is closed")
        return self._handle

    @property
    def torch_dtype(self):
        return _TORCH_DTYPE[self.params.dtype]

    def close(self):
        if self._handle is not None:
            h, self._handle = self._handle, None
            _check(library().hga_plan_destroy(h))

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- calls ---

def hga_build_summaries(plan: Plan, k_rot, chunk_begin: int, chunk_end: int, chunk_sum,
                        group_sum, k_chunk0: int = 0, stream=None):
    """k_rot [B, Hkv, k_tokens, d]; chunk_sum [B, Hkv, table_chunks, d] fp32;
    group_sum [B, Hkv, table_chunks*C/G, d] fp32."""
    _check(library().hga_build_summaries(
        plan.handle, _ptr(k_rot), k_rot.shape[2], k_chunk0, chunk_begin, chunk_end,
        _ptr(chunk_sum), _ptr(group_sum), chunk_sum.shape[2], _stream(stream)))


def hga_route_chunks(plan: Plan, q_rot, q_chunk0: int, chunk_sum, qbar, chunk_idx, stream=None):
    """q_rot [B, Hq, n_q_chunks*C, d]; qbar [B, Hkv, n_q_chunks, d] fp32;
    chunk_idx [B, Hkv, n_q_chunks, K_c] int32."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_route_chunks(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(chunk_sum), chunk_sum.shape[2],
        _ptr(qbar), _ptr(chunk_idx), _stream(stream)))


def hga_route_groups(plan: Plan, qbar, chunk_idx, q_chunk0: int, group_sum, group_idx,
                     stream=None):
    """group_sum [B, Hkv, table_chunks*C/G, d] fp32; group_idx [B, Hkv, n_q_chunks, K_g]."""
    gpc = plan.params.chunk // plan.params.group
    _check(library().hga_route_groups(
        plan.handle, _ptr(qbar), _ptr(chunk_idx), q_chunk0, qbar.shape[2], _ptr(group_sum),
        group_sum.shape[2] // gpc, _ptr(group_idx), _stream(stream)))


def hga_route(plan: Plan, q_rot, q_chunk0: int, chunk_sum, group_sum, qbar, chunk_idx,
              group_idx, stream=None):
    """Both routing stages in one launch; same arguments and outputs as
    hga_route_chunks followed by hga_route_groups."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_route(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(chunk_sum), _ptr(group_sum),
        chunk_sum.shape[2], _ptr(qbar), _ptr(chunk_idx), _ptr(group_idx), _stream(stream)))


def hga_build_summaries_qbar(plan: Plan, k_rot, k_chunk0: int, chunk_begin: int, chunk_end: int,
                             chunk_sum, group_sum, q_rot, q_chunk0: int, qbar, stream=None):
    """hga_build_summaries and the query means of q_rot in one launch."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_build_summaries_qbar(
        plan.handle, _ptr(k_rot), k_rot.shape[2], k_chunk0, chunk_begin, chunk_end,
        _ptr(chunk_sum), _ptr(group_sum), chunk_sum.shape[2], _ptr(q_rot), q_chunk0, nq,
        _ptr(qbar), _stream(stream)))


def hga_route_qbar(plan: Plan, qbar, q_chunk0: int, chunk_sum, group_sum, chunk_idx, group_idx,
                   stream=None):
    """hga_route's selection stages from a given qbar [B, Hkv, n_q_chunks, d]."""
    _check(library().hga_route_qbar(
        plan.handle, _ptr(qbar), q_chunk0, qbar.shape[2], _ptr(chunk_sum), _ptr(group_sum),
        chunk_sum.shape[2], _ptr(chunk_idx), _ptr(group_idx), _stream(stream)))


def hga_gather_kv(plan: Plan, group_idx, q_chunk0: int, k_src, v_src, k_routed, v_routed,
                  src_on_host: bool = False, stream=None):
    """k_src/v_src [B, Hkv, src_tokens, d] (device, or pinned host with
    src_on_host); k_routed/v_routed [B, Hkv, n_q_chunks, K_g*G, d]."""
    _check(library().hga_gather_kv(
        plan.handle, _ptr(group_idx), q_chunk0, group_idx.shape[2], _ptr(k_src), _ptr(v_src),
        k_src.shape[2], int(bool(src_on_host)), _ptr(k_routed), _ptr(v_routed),
        _stream(stream)))


class WarmCache:
    """Device buffers of a warm LRU cache of routed groups (one partition of
    n_slots slots per (batch, KV head)) for hga_gather_kv_cached; every map
    entry starts at -1 (empty)."""

    def __init__(self, plan: Plan, n_slots: int, src_tokens: int, device="cuda"):
        p = plan.params
        bh = (p.batch, p.n_kv_heads)
        dt = _TORCH_DTYPE[p.dtype]
        self.n_slots = n_slots
        self.k = torch.zeros(*bh, n_slots, p.group, p.head_dim, dtype=dt, device=device)
        self.v = torch.zeros_like(self.k)
        i32 = torch.int32
        self.slot_group = torch.full((*bh, n_slots), -1, dtype=i32, device=device)
        self.slot_used = torch.full((*bh, n_slots), -1, dtype=i32, device=device)
        self.map_groups = src_tokens // p.group
        self.group_slot = torch.full((*bh, self.map_groups), -1, dtype=i32, device=device)
        self.entry_slot = torch.empty((*bh, p.topk_groups), dtype=i32, device=device)
        self.tick = 0


def hga_gather_kv_cached(plan: Plan, group_idx, c: int, k_src, v_src, cache: WarmCache,
                         k_routed, v_routed, n_fetched=None, src_on_host: bool = False,
                         stream=None):
    """hga_gather_kv for query chunk c (group_idx [B, Hkv, 1, K_g]) through
    `cache`; the call's tick is cache.tick, which is then advanced."""
    _check(library().hga_gather_kv_cached(
        plan.handle, _ptr(group_idx), c, _ptr(k_src), _ptr(v_src), k_src.shape[2],
        int(bool(src_on_host)), _ptr(cache.k), _ptr(cache.v), cache.n_slots,
        _ptr(cache.slot_group), _ptr(cache.slot_used), _ptr(cache.group_slot),
        cache.map_groups, _ptr(cache.entry_slot), cache.tick,
        _ptr(k_routed), _ptr(v_routed), _ptr(n_fetched), _stream(stream)))
    cache.tick += 1


def hga_attend(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, k_routed, v_routed, group_idx,
               out, lse=None, res_slot=None, stream=None):
    """q_rot/out [B, Hq, n_q_chunks*C, d]; k_res/v_res [B, Hkv, res_tokens, d];
    lse [B, Hq, n_q_chunks*C] fp32 or None; res_slot int32 or None."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_attend(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(res_slot), _ptr(k_routed), _ptr(v_routed), _ptr(group_idx), _ptr(out), _ptr(lse),
        _stream(stream)))


def hga_attend_timed(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, k_routed, v_routed,
                     group_idx, out, start_event, stop_event, lse=None, res_slot=None,
                     stream=None):
    """hga_attend whose kernel dispatch records the two events (torch.cuda.Event
    objects that have been recorded once, so that they exist)."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_attend_timed(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(res_slot), _ptr(k_routed), _ptr(v_routed), _ptr(group_idx), _ptr(out), _ptr(lse),
        start_event.cuda_event, stop_event.cuda_event, _stream(stream)))


def hga_attend_split_workspace(plan: Plan, n_q_chunks: int) -> int:
    """Bytes of workspace hga_attend_split uses at most for n_q_chunks chunks."""
    n = library().hga_attend_split_workspace(plan.handle, n_q_chunks)
    if n < 0:
        raise HgaError(-1, "hga_attend_split_workspace: invalid plan or n_q_chunks")
    return n


def hga_attend_split(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, k_routed, v_routed,
                     group_idx, out, workspace, lse=None, res_slot=None, stream=None):
    """hga_attend with each unit's key tiles spread over several workgroups;
    workspace: a device tensor (any dtype) of at least
    hga_attend_split_workspace bytes for the most splits, or None."""
    nq = q_rot.shape[2] // plan.params.chunk
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(library().hga_attend_split(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(res_slot), _ptr(k_routed), _ptr(v_routed), _ptr(group_idx), _ptr(out), _ptr(lse),
        _ptr(workspace), nbytes, _stream(stream)))


def hga_attend_split_static(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, k_routed, v_routed,
                            group_idx, out, lse=None, res_slot=None, stream=None):
    """hga_attend_split with the library's static per-device scratch as the
    workspace: allocates nothing."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_attend_split_static(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(res_slot), _ptr(k_routed), _ptr(v_routed), _ptr(group_idx), _ptr(out), _ptr(lse),
        _stream(stream)))


def hga_static_scratch_bytes() -> int:
    """Size of the per-device array hga_attend_split_static uses."""
    return library().hga_static_scratch_bytes()


def hga_gather_attend_split(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, k_src, v_src,
                            group_idx, k_routed, v_routed, out, workspace, lse=None,
                            res_slot=None, src_on_host=False, stream=None):
    """hga_gather_kv (from k_src/v_src [B, Hkv, src_tokens, d], device or
    pinned host) + hga_attend_split in one pass; k_routed/v_routed written
    (or both None: gathered on chip only)."""
    nq = q_rot.shape[2] // plan.params.chunk
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(library().hga_gather_attend_split(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(res_slot), _ptr(k_src), _ptr(v_src), k_src.shape[2], 1 if src_on_host else 0,
        _ptr(group_idx), _ptr(k_routed), _ptr(v_routed), _ptr(out), _ptr(lse),
        _ptr(workspace), nbytes, _stream(stream)))


def hga_attend_backward(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, group_idx, out, lse,
                        dout, dq, dk, dv, stream=None):
    """Gradients of hga_attend (bf16, prefill layout): dq [B, Hq, nq*C, d]
    fp32 written; dk, dv [B, Hkv, res_tokens, d] fp32 added into."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_attend_backward(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(group_idx), _ptr(out), _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
        _stream(stream)))


def hga_gather_attend(plan: Plan, q_rot, q_chunk0: int, k_res, v_res, group_idx, k_routed,
                      v_routed, out, lse=None, start_event=None, stop_event=None, stream=None):
    """hga_gather_kv + hga_attend in one pass (prefill layout: k_res/v_res
    [B, Hkv, res_tokens, d] indexed by token); k_routed/v_routed
    [B, Hkv, n_q_chunks, K_g*G, d] are written, or both None: the routed rows
    are gathered on chip only.  start/stop_event: recorded torch.cuda.Event
    objects or None."""
    nq = q_rot.shape[2] // plan.params.chunk
    _check(library().hga_gather_attend(
        plan.handle, _ptr(q_rot), q_chunk0, nq, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(group_idx), _ptr(k_routed), _ptr(v_routed), _ptr(out), _ptr(lse),
        start_event.cuda_event if start_event is not None else None,
        stop_event.cuda_event if stop_event is not None else None, _stream(stream)))


def _ws(workspace):
    return (_ptr(workspace),
            workspace.numel() * workspace.element_size() if workspace is not None else 0)


def hga_block_step(plan: Plan, q_block, c: int, k_res, v_res, chunk_sum, group_sum, qbar,
                   chunk_idx, group_idx, k_routed, v_routed, out, lse=None, workspace=None,
                   stream=None):
    """One block of a block-sequential prefill: route query chunk c, gather +
    attend it, append chunk c's summaries.  q_block/out [B, Hq, C, d];
    k_res/v_res [B, Hkv, res_tokens, d]; the per-chunk outputs have a
    query-chunk dimension of 1.  workspace: None (bit-identical to the bulk
    prefill) or a device tensor for the split attention."""
    _check(library().hga_block_step(
        plan.handle, _ptr(q_block), c, _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(chunk_sum), _ptr(group_sum), chunk_sum.shape[2], _ptr(qbar), _ptr(chunk_idx),
        _ptr(group_idx), _ptr(k_routed), _ptr(v_routed), _ptr(out), _ptr(lse), *_ws(workspace),
        _stream(stream)))


def hga_prefill_blocks(plan: Plan, q_blocks, k_res, v_res, chunk_sum, group_sum, qbar,
                       chunk_idx, group_idx, k_routed, v_routed, out, lse=None, workspace=None,
                       stream=None):
    """hga_block_step for blocks 0 .. n_blocks-1 in order; block-major
    buffers (first dimension n_blocks); workspace as for hga_block_step."""
    _check(library().hga_prefill_blocks(
        plan.handle, _ptr(q_blocks), q_blocks.shape[0], _ptr(k_res), _ptr(v_res), k_res.shape[2],
        _ptr(chunk_sum), _ptr(group_sum), chunk_sum.shape[2], _ptr(qbar), _ptr(chunk_idx),
        _ptr(group_idx), _ptr(k_routed), _ptr(v_routed), _ptr(out), _ptr(lse), *_ws(workspace),
        _stream(stream)))
