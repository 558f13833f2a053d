"""Device buffers and the five-call sequence for one workload.

``PrefillPipeline``: every token's K/V is resident in device memory; one step
summarises every chunk, routes every query chunk, gathers the routed groups
(device to device) and attends.

``DecodePipeline``: the history K/V lives in pinned host memory (the paper's
RAM-backed cold tier, Sec. 4.3); the device holds the summary tables, the
always-visible first and recent chunks and the current 64-token block.  One
step routes the block, gathers only its routed groups over the host link,
attends (``hga_attend_split``; or both in one call,
``hga_gather_attend_split``, with ``fused_gather=True``), and appends the
block's summaries (the store's "append").

Prefill routing has three equivalent forms (bit-identical summaries, query
means and indices), chosen by ``route_mode``: "fused" (``hga_build_summaries``
then ``hga_route``), "separate" (``hga_route_chunks`` then
``hga_route_groups``), and "qbar" (``hga_build_summaries_qbar``, which also
reduces the query means in the same launch, then ``hga_route_qbar``).  The
gather and the attention are either one call, ``hga_gather_attend``
(``gather_mode="fused"``, the default: the attention stages the routed rows
from the resident K/V and writes the routed buffers), or the two calls
``hga_gather_kv`` and ``hga_attend`` (``gather_mode="separate"``); the
results are identical.  Both pipelines only allocate with torch and call the
binding; all arithmetic runs in the HIP library.
"""

from __future__ import annotations

import numpy as np
import torch

from . import hga

__all__ = ["PrefillPipeline", "BlockPrefillPipeline", "DecodePipeline", "to_device"]


def to_device(arr: np.ndarray, dtype: str, device="cuda", pin=False) -> torch.Tensor:
    """Storage array from the workload generator -> torch tensor with the same bytes."""
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if dtype == "bf16":
        t = t.view(torch.bfloat16)
    if pin:
        return t.pin_memory()
    return t.to(device)


class PrefillPipeline:
    def __init__(self, w, inputs: dict, device="cuda", plan: hga.Plan | None = None,
                 route_mode: str = "qbar", gather_mode: str = "fused", routed_out: bool = True):
        """routed_out: with the fused gather, also write the gathered rows to
        k_routed/v_routed (False: they stay on chip; the separate gather
        always writes them)."""
        assert not w.decode_block
        assert route_mode in ("fused", "separate", "qbar")
        assert gather_mode in ("fused", "separate")
        self.w = w
        self.route_mode = route_mode
        self.gather_mode = gather_mode
        self.routed_out = routed_out or gather_mode == "separate"
        self.plan = plan or hga.Plan.for_workload(w)
        B, Hkv, d, C, G = w.batch, w.n_kv_heads, w.head_dim, w.chunk, w.group
        nc = w.n_chunks
        f32, i32 = torch.float32, torch.int32
        self.q = to_device(inputs["q"], w.dtype, device)
        self.k = to_device(inputs["k"], w.dtype, device)
        self.v = to_device(inputs["v"], w.dtype, device)
        dt = self.q.dtype
        self.chunk_sum = torch.empty(B, Hkv, nc, d, dtype=f32, device=device)
        self.group_sum = torch.empty(B, Hkv, nc * (C // G), d, dtype=f32, device=device)
        self.qbar = torch.empty(B, Hkv, nc, d, dtype=f32, device=device)
        self.chunk_idx = torch.empty(B, Hkv, nc, w.topk_chunks, dtype=i32, device=device)
        self.group_idx = torch.empty(B, Hkv, nc, w.topk_groups, dtype=i32, device=device)
        self.k_routed = torch.empty(B, Hkv, nc, w.topk_groups * G, d, dtype=dt, device=device)
        self.v_routed = torch.empty_like(self.k_routed)
        self.out = torch.empty_like(self.q)
        self.lse = torch.empty(B, w.n_q_heads, w.seq_len, dtype=f32, device=device)

    def summaries(self, stream=None):
        if self.route_mode == "qbar":
            hga.hga_build_summaries_qbar(self.plan, self.k, 0, 0, self.w.n_chunks,
                                         self.chunk_sum, self.group_sum, self.q, 0, self.qbar,
                                         stream=stream)
            return
        hga.hga_build_summaries(self.plan, self.k, 0, self.w.n_chunks, self.chunk_sum,
                                self.group_sum, stream=stream)

    def route(self, stream=None):
        if self.route_mode == "qbar":
            hga.hga_route_qbar(self.plan, self.qbar, 0, self.chunk_sum, self.group_sum,
                               self.chunk_idx, self.group_idx, stream=stream)
            return
        if self.route_mode == "fused":
            hga.hga_route(self.plan, self.q, 0, self.chunk_sum, self.group_sum, self.qbar,
                          self.chunk_idx, self.group_idx, stream=stream)
            return
        hga.hga_route_chunks(self.plan, self.q, 0, self.chunk_sum, self.qbar, self.chunk_idx,
                             stream=stream)
        hga.hga_route_groups(self.plan, self.qbar, self.chunk_idx, 0, self.group_sum,
                             self.group_idx, stream=stream)

    def gather(self, stream=None):
        hga.hga_gather_kv(self.plan, self.group_idx, 0, self.k, self.v, self.k_routed,
                          self.v_routed, stream=stream)

    def attend(self, stream=None):
        hga.hga_attend(self.plan, self.q, 0, self.k, self.v, self.k_routed, self.v_routed,
                       self.group_idx, self.out, self.lse, stream=stream)

    def gather_attend(self, stream=None, start_event=None, stop_event=None):
        kr, vr = (self.k_routed, self.v_routed) if self.routed_out else (None, None)
        hga.hga_gather_attend(self.plan, self.q, 0, self.k, self.v, self.group_idx, kr, vr,
                              self.out, self.lse, start_event=start_event,
                              stop_event=stop_event, stream=stream)

    def backward(self, dout, stream=None):
        """Gradients of the attention of the last ``step`` for output gradient
        ``dout`` (like ``out``): returns (dq, dk, dv), fp32, dk and dv in
        the resident K/V layout (routing held fixed)."""
        dq = torch.empty(self.q.shape, dtype=torch.float32, device=self.q.device)
        dk = torch.zeros(self.k.shape, dtype=torch.float32, device=self.k.device)
        dv = torch.zeros_like(dk)
        hga.hga_attend_backward(self.plan, self.q, 0, self.k, self.v, self.group_idx, self.out,
                                self.lse, dout, dq, dk, dv, stream=stream)
        return dq, dk, dv

    def step(self, stream=None):
        self.summaries(stream)
        self.route(stream)
        if self.gather_mode == "fused":
            self.gather_attend(stream)
        else:
            self.gather(stream)
            self.attend(stream)


class BlockPrefillPipeline:
    """The prompt processed as a sequence of 64-token blocks, each routed
    against the summaries of the chunks closed before it, attended, and then
    appended to the tables (``hga_prefill_blocks``: one native loop of
    ``hga_block_step``).  Queries, outputs and the per-block routing results
    are block-major ([n_blocks, ...]); K/V are the whole prompt's,
    token-indexed, as in the bulk prefill.  ``split_attend``: the blocks'
    attention in its split form (a workspace spreads each block's few units
    over more workgroups); without it every output is bit-identical to the
    bulk prefill's."""

    def __init__(self, w, inputs: dict, device="cuda", plan: hga.Plan | None = None,
                 split_attend: bool = False):
        assert not w.decode_block
        self.w = w
        self.plan = plan or hga.Plan.for_workload(w)
        B, Hq, Hkv, d, C, G = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.chunk, w.group
        nc = w.n_chunks
        f32, i32 = torch.float32, torch.int32
        q = np.ascontiguousarray(
            inputs["q"].reshape(B, Hq, nc, C, d).transpose(2, 0, 1, 3, 4))
        self.q_blocks = to_device(q, w.dtype, device)            # [nc, B, Hq, C, d]
        self.k = to_device(inputs["k"], w.dtype, device)
        self.v = to_device(inputs["v"], w.dtype, device)
        dt = self.k.dtype
        self.chunk_sum = torch.zeros(B, Hkv, nc, d, dtype=f32, device=device)
        self.group_sum = torch.zeros(B, Hkv, nc * (C // G), d, dtype=f32, device=device)
        self.qbar = torch.empty(nc, B, Hkv, 1, d, dtype=f32, device=device)
        self.chunk_idx = torch.empty(nc, B, Hkv, 1, w.topk_chunks, dtype=i32, device=device)
        self.group_idx = torch.empty(nc, B, Hkv, 1, w.topk_groups, dtype=i32, device=device)
        self.k_routed = torch.empty(nc, B, Hkv, 1, w.topk_groups * G, d, dtype=dt, device=device)
        self.v_routed = torch.empty_like(self.k_routed)
        self.out = torch.empty_like(self.q_blocks)
        self.lse = torch.empty(nc, B, Hq, C, dtype=f32, device=device)
        self.attend_ws = None
        if split_attend:
            nbytes = hga.hga_attend_split_workspace(self.plan, 1)
            self.attend_ws = torch.empty((nbytes + 3) // 4, dtype=f32, device=device)

    def step(self, stream=None):
        hga.hga_prefill_blocks(self.plan, self.q_blocks, self.k, self.v, self.chunk_sum,
                               self.group_sum, self.qbar, self.chunk_idx, self.group_idx,
                               self.k_routed, self.v_routed, self.out, self.lse,
                               workspace=self.attend_ws, stream=stream)


class DecodePipeline:
    """One query block (the last chunk of the workload) after a host-resident history."""

    def __init__(self, w, inputs: dict, device="cuda", plan: hga.Plan | None = None,
                 fused_route: bool = True, split_attend: bool = True, fused_gather: bool = False,
                 qbar_first: bool = True):
        assert w.decode_block and w.decode_blocks == 1
        self.w = w
        self.fused_route = fused_route
        # qbar_first: the block's summaries and its q_bar in one launch
        # (hga_build_summaries_qbar) before routing from q_bar
        # (hga_route_qbar), so the routing launch does not wait on the query
        # rows; the block's own chunk is never among its routing candidates.
        # Otherwise hga_route forms q_bar and the summaries follow the block.
        self.qbar_first = qbar_first and fused_route
        # fused_gather: the host gather inside the split attention
        # (hga_gather_attend_split), else hga_gather_kv then the attention.
        # The separate gather is the faster one here: each unit's two query
        # workgroups would both pull its routed rows over the host link.
        self.fused_gather = fused_gather and split_attend
        self.plan = plan or hga.Plan.for_workload(w)
        B, Hkv, d, C, G = w.batch, w.n_kv_heads, w.head_dim, w.chunk, w.group
        f32, i32 = torch.float32, torch.int32
        c = w.q_chunk0                      # the block's chunk id
        self.c = c
        hist = c * C
        k_all = to_device(inputs["k"], w.dtype, "cpu")
        v_all = to_device(inputs["v"], w.dtype, "cpu")
        # cold tier: the history in pinned host memory
        self.k_hist = k_all[:, :, :hist].contiguous().pin_memory()
        self.v_hist = v_all[:, :, :hist].contiguous().pin_memory()
        # hot tier: the chunks the block sees besides its own (the library's
        # visibility rule: first F chunks, the recent window), then the block
        hot = hga.hga_visible_chunks(self.plan.params, c)
        self.hot_chunks = hot + [c]
        slot = np.full(c + 1, -1, dtype=np.int32)
        for s, cc in enumerate(self.hot_chunks):
            slot[cc] = s
        self.res_slot = torch.from_numpy(slot).to(device)
        idx = torch.tensor([t for cc in self.hot_chunks for t in range(cc * C, (cc + 1) * C)])
        self.k_res = k_all[:, :, idx].contiguous().to(device)
        self.v_res = v_all[:, :, idx].contiguous().to(device)
        self.cur_slot = len(hot)
        dt = self.k_res.dtype
        self.q = to_device(inputs["q"], w.dtype, device)           # [B, Hq, 64, d]
        self.table_chunks = c + 1
        self.chunk_sum = torch.zeros(B, Hkv, c + 1, d, dtype=f32, device=device)
        self.group_sum = torch.zeros(B, Hkv, (c + 1) * (C // G), d, dtype=f32, device=device)
        self.qbar = torch.empty(B, Hkv, 1, d, dtype=f32, device=device)
        self.chunk_idx = torch.empty(B, Hkv, 1, w.topk_chunks, dtype=i32, device=device)
        self.group_idx = torch.empty(B, Hkv, 1, w.topk_groups, dtype=i32, device=device)
        self.k_routed = torch.empty(B, Hkv, 1, w.topk_groups * G, d, dtype=dt, device=device)
        self.v_routed = torch.empty_like(self.k_routed)
        self.out = torch.empty_like(self.q)
        self.lse = torch.empty(B, w.n_q_heads, C, dtype=f32, device=device)
        # The block's four units would leave most of the chip idle in one
        # workgroup each: hga_attend_split spreads their key tiles (its
        # partial results live in this workspace, allocated once).
        self.attend_ws = None
        if split_attend:
            nbytes = hga.hga_attend_split_workspace(self.plan, 1)
            self.attend_ws = torch.empty((nbytes + 3) // 4, dtype=f32, device=device)
        # The history's summaries were appended as its chunks closed; build
        # them once here from a transient device copy of the history keys.
        k_dev = self.k_hist.to(device)
        hga.hga_build_summaries(self.plan, k_dev, 0, c, self.chunk_sum, self.group_sum)
        torch.cuda.synchronize()
        del k_dev

    def pcie_bytes_per_step(self) -> int:
        """Bytes the gather pulls across the host link: K and V of every valid routed group."""
        n = int((self.group_idx >= 0).sum().item())
        return 2 * n * self.w.group * self.w.head_dim * self.w.elem_bytes

    def route(self, stream=None):
        if self.fused_route:
            hga.hga_route(self.plan, self.q, self.c, self.chunk_sum, self.group_sum, self.qbar,
                          self.chunk_idx, self.group_idx, stream=stream)
            return
        hga.hga_route_chunks(self.plan, self.q, self.c, self.chunk_sum, self.qbar,
                             self.chunk_idx, stream=stream)
        hga.hga_route_groups(self.plan, self.qbar, self.chunk_idx, self.c, self.group_sum,
                             self.group_idx, stream=stream)

    def gather(self, stream=None):
        hga.hga_gather_kv(self.plan, self.group_idx, self.c, self.k_hist, self.v_hist,
                          self.k_routed, self.v_routed, src_on_host=True, stream=stream)

    def attend(self, stream=None):
        if self.attend_ws is not None:
            hga.hga_attend_split(self.plan, self.q, self.c, self.k_res, self.v_res,
                                 self.k_routed, self.v_routed, self.group_idx, self.out,
                                 self.attend_ws, self.lse, res_slot=self.res_slot, stream=stream)
            return
        hga.hga_attend(self.plan, self.q, self.c, self.k_res, self.v_res, self.k_routed,
                       self.v_routed, self.group_idx, self.out, self.lse,
                       res_slot=self.res_slot, stream=stream)

    def append(self, stream=None):
        """Summaries of the block's chunk once it closes (store "append")."""
        # k_res row cur_slot*C is the block's first token: chunk c sits at
        # chunk offset cur_slot of the resident buffer.
        hga.hga_build_summaries(self.plan, self.k_res, self.c, self.c + 1, self.chunk_sum,
                                self.group_sum, k_chunk0=self.c - self.cur_slot, stream=stream)

    def gather_attend(self, stream=None):
        """The routed groups copied from pinned host memory by the split
        attention's own workgroups while the others attend the resident chunks."""
        hga.hga_gather_attend_split(self.plan, self.q, self.c, self.k_res, self.v_res,
                                    self.k_hist, self.v_hist, self.group_idx, self.k_routed,
                                    self.v_routed, self.out, self.attend_ws, self.lse,
                                    res_slot=self.res_slot, src_on_host=True, stream=stream)

    def append_qbar(self, stream=None):
        """The block's chunk summaries (as ``append``) and its q_bar, one launch."""
        hga.hga_build_summaries_qbar(self.plan, self.k_res, self.c - self.cur_slot, self.c,
                                     self.c + 1, self.chunk_sum, self.group_sum, self.q, self.c,
                                     self.qbar, stream=stream)

    def step(self, stream=None):
        if self.qbar_first:
            self.append_qbar(stream)
            hga.hga_route_qbar(self.plan, self.qbar, self.c, self.chunk_sum, self.group_sum,
                               self.chunk_idx, self.group_idx, stream=stream)
        else:
            self.route(stream)
        if self.fused_gather:
            self.gather_attend(stream)
        else:
            self.gather(stream)
            self.attend(stream)
        if not self.qbar_first:
            self.append(stream)


class DecodeSequencePipeline:
    """Consecutive 64-token decode blocks (the last ``w.decode_blocks`` chunks)
    after a host-resident history, each routed, gathered, attended and then
    appended before the next one, as a serving loop does.

    The history K/V of the whole sequence lives in pinned host memory (only
    chunks before the current block are ever read).  The device holds the
    sink chunks and, compactly, every block's recent window and current
    chunk (``res_slot`` maps chunk -> slot), the summary tables (built for
    the history once, then appended block by block) and, with
    ``cache_slots``, a warm LRU cache of routed groups (``hga.WarmCache``):
    a routed group still in the cache is copied from device memory, only the
    others cross the host link.  Without a cache every block's routed groups
    come from host memory (``hga_gather_kv``)."""

    def __init__(self, w, inputs: dict, device="cuda", plan: hga.Plan | None = None,
                 cache_slots: int | None = None, qbar_first: bool = True):
        assert w.decode_block
        self.w = w
        self.qbar_first = qbar_first  # as DecodePipeline's
        self.plan = plan or hga.Plan.for_workload(w)
        B, Hq, Hkv, d, C, G = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.chunk, w.group
        f32, i32 = torch.float32, torch.int32
        self.c0, self.n_blocks = w.q_chunk0, w.decode_blocks
        c_end = self.c0 + self.n_blocks
        k_all = to_device(inputs["k"], w.dtype, "cpu")
        v_all = to_device(inputs["v"], w.dtype, "cpu")
        self.k_hist = k_all.contiguous().pin_memory()      # cold tier: every token
        self.v_hist = v_all.contiguous().pin_memory()
        # hot tier: every chunk some block sees besides its own (the
        # library's visibility rule), and the blocks' own chunks
        hot = sorted(set(range(self.c0, c_end)).union(
            *(hga.hga_visible_chunks(self.plan.params, c) for c in range(self.c0, c_end))))
        slot = np.full(c_end, -1, dtype=np.int32)
        for s, cc in enumerate(hot):
            slot[cc] = s
        self.slot_of = slot
        self.res_slot = torch.from_numpy(slot).to(device)
        idx = torch.tensor([t for cc in hot for t in range(cc * C, (cc + 1) * C)])
        self.k_res = k_all[:, :, idx].contiguous().to(device)
        self.v_res = v_all[:, :, idx].contiguous().to(device)
        dt = self.k_res.dtype
        q = to_device(inputs["q"], w.dtype, "cpu")           # [B, Hq, n_blocks*C, d]
        self.q_blocks = q.reshape(B, Hq, self.n_blocks, C, d).permute(2, 0, 1, 3, 4) \
            .contiguous().to(device)                          # [n_blocks, B, Hq, C, d]
        self.chunk_sum = torch.zeros(B, Hkv, c_end, d, dtype=f32, device=device)
        self.group_sum = torch.zeros(B, Hkv, c_end * (C // G), d, dtype=f32, device=device)
        self.qbar = torch.empty(B, Hkv, 1, d, dtype=f32, device=device)
        self.chunk_idx = torch.empty(B, Hkv, 1, w.topk_chunks, dtype=i32, device=device)
        self.group_idx = torch.empty(self.n_blocks, B, Hkv, 1, w.topk_groups, dtype=i32,
                                     device=device)
        self.k_routed = torch.empty(B, Hkv, 1, w.topk_groups * G, d, dtype=dt, device=device)
        self.v_routed = torch.empty_like(self.k_routed)
        self.out = torch.empty_like(self.q_blocks)
        self.lse = torch.empty(self.n_blocks, B, Hq, C, dtype=f32, device=device)
        self.n_fetched = torch.zeros(self.n_blocks, B, Hkv, dtype=i32, device=device)
        nbytes = hga.hga_attend_split_workspace(self.plan, 1)
        self.attend_ws = torch.empty((nbytes + 3) // 4, dtype=f32, device=device)
        self.cache = (hga.WarmCache(self.plan, cache_slots, self.k_hist.shape[2], device)
                      if cache_slots else None)
        # the history's summaries, built once from a transient device copy
        k_dev = self.k_hist[:, :, :self.c0 * C].to(device)
        hga.hga_build_summaries(self.plan, k_dev, 0, self.c0, self.chunk_sum, self.group_sum)
        torch.cuda.synchronize()
        del k_dev

    def block(self, b: int, stream=None):
        """Route, gather, attend and append block b (query chunk c0 + b)."""
        c = self.c0 + b
        q = self.q_blocks[b]
        gi = self.group_idx[b]
        k_chunk0 = c - int(self.slot_of[c])  # chunk c sits at resident slot slot_of[c]
        if self.qbar_first:
            hga.hga_build_summaries_qbar(self.plan, self.k_res, k_chunk0, c, c + 1,
                                         self.chunk_sum, self.group_sum, q, c, self.qbar,
                                         stream=stream)
            hga.hga_route_qbar(self.plan, self.qbar, c, self.chunk_sum, self.group_sum,
                               self.chunk_idx, gi, stream=stream)
        else:
            hga.hga_route(self.plan, q, c, self.chunk_sum, self.group_sum, self.qbar,
                          self.chunk_idx, gi, stream=stream)
        if self.cache is not None:
            hga.hga_gather_kv_cached(self.plan, gi, c, self.k_hist, self.v_hist, self.cache,
                                     self.k_routed, self.v_routed, self.n_fetched[b],
                                     src_on_host=True, stream=stream)
        else:
            hga.hga_gather_kv(self.plan, gi, c, self.k_hist, self.v_hist, self.k_routed,
                              self.v_routed, src_on_host=True, stream=stream)
        hga.hga_attend_split(self.plan, q, c, self.k_res, self.v_res, self.k_routed,
                             self.v_routed, gi, self.out[b], self.attend_ws, self.lse[b],
                             res_slot=self.res_slot, stream=stream)
        if not self.qbar_first:
            # chunk c closes: its summaries from the resident copy
            hga.hga_build_summaries(self.plan, self.k_res, c, c + 1, self.chunk_sum,
                                    self.group_sum, k_chunk0=k_chunk0, stream=stream)

    def step_overlapped(self, copy_stream=None):
        """All blocks, with each block's gather (the warm cache's bookkeeping
        and copies, the misses over the host link) on `copy_stream` while the
        previous block attends on the current stream (Sec. 4.3: the cold tier
        feeds the warm one while the hot set computes).  Same calls and
        results as ``step`` (routing, routed rows, outputs, cache maps): the
        current stream runs block b+1's summaries and routing before block b's
        attention; events order gather(b) after routing(b) and before
        attention(b), and gather(b+2) after attention(b), whose routed buffers
        (two sets, alternating) it overwrites.  Requires ``qbar_first`` (the
        block's own chunk summarised before it routes)."""
        assert self.qbar_first
        main = torch.cuda.current_stream()
        side = copy_stream or self._copy_stream()
        if not hasattr(self, "k_routed2"):
            self.k_routed2 = torch.empty((2, *self.k_routed.shape), dtype=self.k_routed.dtype,
                                         device=self.k_routed.device)
            self.v_routed2 = torch.empty_like(self.k_routed2)
        ev_route = [torch.cuda.Event() for _ in range(self.n_blocks)]
        ev_gather = [torch.cuda.Event() for _ in range(self.n_blocks)]
        ev_attend = [torch.cuda.Event() for _ in range(self.n_blocks)]

        def route(b):
            c = self.c0 + b
            k_chunk0 = c - int(self.slot_of[c])
            hga.hga_build_summaries_qbar(self.plan, self.k_res, k_chunk0, c, c + 1,
                                         self.chunk_sum, self.group_sum, self.q_blocks[b], c,
                                         self.qbar, stream=main)
            hga.hga_route_qbar(self.plan, self.qbar, c, self.chunk_sum, self.group_sum,
                               self.chunk_idx, self.group_idx[b], stream=main)
            ev_route[b].record(main)

        def gather(b):
            c = self.c0 + b
            side.wait_event(ev_route[b])
            if b >= 2:
                side.wait_event(ev_attend[b - 2])
            kr, vr = self.k_routed2[b % 2], self.v_routed2[b % 2]
            if self.cache is not None:
                hga.hga_gather_kv_cached(self.plan, self.group_idx[b], c, self.k_hist,
                                         self.v_hist, self.cache, kr, vr, self.n_fetched[b],
                                         src_on_host=True, stream=side)
            else:
                hga.hga_gather_kv(self.plan, self.group_idx[b], c, self.k_hist, self.v_hist, kr,
                                  vr, src_on_host=True, stream=side)
            ev_gather[b].record(side)

        def attend(b):
            c = self.c0 + b
            main.wait_event(ev_gather[b])
            hga.hga_attend_split(self.plan, self.q_blocks[b], c, self.k_res, self.v_res,
                                 self.k_routed2[b % 2], self.v_routed2[b % 2], self.group_idx[b],
                                 self.out[b], self.attend_ws, self.lse[b],
                                 res_slot=self.res_slot, stream=main)
            ev_attend[b].record(main)

        route(0)
        gather(0)
        for b in range(self.n_blocks):
            if b + 1 < self.n_blocks:
                route(b + 1)
                gather(b + 1)
            attend(b)
        # the copy stream's work is joined before the caller's next use
        main.wait_event(ev_gather[self.n_blocks - 1])

    def capture(self, overlapped: bool = True):
        """One step (all blocks) recorded as a HIP graph: replaying it
        launches every block's kernels, and with `overlapped` the two-stream
        schedule of ``step_overlapped`` with its stream joins as graph edges
        instead of event waits.  The calls' arguments are fixed at capture
        (the warm cache's ticks included), so a replay is the step of a fresh
        sequence after ``reset_cache``.  No call captured here records a
        memset node."""
        self.reset_cache()
        (self.step_overlapped if overlapped else self.step)()   # warm-up, eager
        torch.cuda.synchronize()
        self.reset_cache()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            (self.step_overlapped if overlapped else self.step)()
        torch.cuda.synchronize()
        return g

    def _copy_stream(self):
        if not hasattr(self, "_side"):
            self._side = torch.cuda.Stream()   # default priority
        return self._side

    def reset_cache(self):
        """Empty the warm cache (a new sequence); its tick keeps counting."""
        if self.cache is not None:
            for t in (self.cache.slot_group, self.cache.slot_used, self.cache.group_slot):
                t.fill_(-1)

    def step(self, stream=None):
        for b in range(self.n_blocks):
            self.block(b, stream)

    def pcie_bytes(self) -> int:
        """Bytes that crossed the host link for the blocks' routed groups."""
        w = self.w
        row = w.head_dim * w.elem_bytes
        if self.cache is not None:
            return int(self.n_fetched.sum().item()) * 2 * w.group * row
        return int((self.group_idx >= 0).sum().item()) * 2 * w.group * row
