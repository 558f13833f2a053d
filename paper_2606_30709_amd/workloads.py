"""Seeded synthetic workloads for the routed-attention path.

This module only *creates inputs*: it draws Gaussian tensors, applies the
model's rotary position embedding to Q and K (the inputs of the routed path
are already-rotated queries and keys, Sec. 2 "RoPE" and Sec. 4.1), plants
"needle" correlations, and rounds to the storage dtype.  It contains none of
the routing method's arithmetic (no summaries, scores, selection or
attention), so both the float64 oracle and the HIP path can consume its bytes.

The presets mirror the paper's shapes:

* ``tiny``      B1 H1/1 d64 N1024 fp32 (oracle-sized prefill)
* ``smalllm``   B4 H8/8 d64 N8192 bf16 (the 40M SmallLM head shape, Sec. 4.2;
  sequence length of the copy-only study, Sec. 5.6)
* ``train12k``  B8 H12/12 d64 N12288 bf16 (the 12,288-token speed study,
  Sec. 5.8), Q/K pre-scaled by 1/sqrt(d)
* ``qwen32k``   B1 H32/4 d128 N32768 bf16, RoPE base 1e6 (Qwen3-30B-A3B
  attention shape, Sec. 4.1), history resident in device memory
* ``decode64k`` one 64-token query block after 65,536 history tokens at the
  Qwen3 shape (the 64K needle-in-a-haystack setting, Sec. 5.3), history in
  pinned host memory
* ``qwen32k_chunks`` the qwen32k shape with the chunk-only routing variant
  of the exact-token Qwen3 wrapper (Sec. 4.1: 16 chunks routed, every group
  of each opened; two sink and eight recent chunks)

Draw order for every preset (seed recorded in the returned dict): raw Q, raw
K, V, then needle placements, then needle directions.  RoPE is applied in
float64, needles are added to the rotated values, and the result is rounded
to fp32 (RNE) and, for bf16 presets, then to bf16 (RNE).
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass

import numpy as np

__all__ = ["Workload", "PRESETS", "preset", "generate", "bf16_bits_to_f64",
           "storage_to_f64", "f64_to_bf16_bits"]


@dataclass(frozen=True)
class Workload:
    key: str
    number: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    seq_len: int              # tokens whose K/V exist (history + query block)
    dtype: str                # "f32" | "bf16"
    rope_base: float
    chunk: int = 64
    group: int = 16
    keep_first: int = 1
    keep_last: int = 0
    force_prev: int = 1
    topk_chunks: int = 2
    topk_groups: int = 4
    prescale: float = 1.0     # multiplies raw Q and K before RoPE
    needle_mode: str = "none"  # "none" | "tail" | "pairs" | "depths"
    needle_count: int = 0
    needle_shift: float = 0.0
    needle_depths: tuple = ()  # chunk ids for needle_mode == "depths"
    decode_block: bool = False  # True: queries are only the last chunk(s)
    decode_blocks: int = 1      # with decode_block: the last this many chunks are query blocks
    rope_wrap: int = 0          # > 0: RoPE positions taken modulo this (Sec. 5, positional
                                # encoding: p mod 65536); a multiple of chunk
    seed: int = 0

    @property
    def n_chunks(self) -> int:
        return self.seq_len // self.chunk

    @property
    def q_chunk0(self) -> int:
        """Absolute id of the first query chunk."""
        return self.n_chunks - self.decode_blocks if self.decode_block else 0

    @property
    def n_q_chunks(self) -> int:
        return self.n_chunks - self.q_chunk0

    @property
    def gqa_ratio(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


PRESETS = {
    "tiny": Workload(
        key="tiny", number=1, batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64,
        seq_len=1024, dtype="f32", rope_base=1e4, keep_first=1, keep_last=0,
        topk_chunks=2, topk_groups=4, needle_mode="tail", needle_count=2,
        needle_shift=2.0, seed=1001),
    "smalllm": Workload(
        key="smalllm", number=2, batch=4, n_q_heads=8, n_kv_heads=8, head_dim=64,
        seq_len=8192, dtype="bf16", rope_base=1e4, keep_first=1, keep_last=0,
        topk_chunks=3, topk_groups=4, needle_mode="pairs", needle_count=8,
        needle_shift=1.5, seed=1002),
    "train12k": Workload(
        key="train12k", number=3, batch=8, n_q_heads=12, n_kv_heads=12,
        head_dim=64, seq_len=12288, dtype="bf16", rope_base=1e4, keep_first=1,
        keep_last=0, topk_chunks=8, topk_groups=12, prescale=0.125, seed=1003),
    "qwen32k": Workload(
        key="qwen32k", number=4, batch=1, n_q_heads=32, n_kv_heads=4,
        head_dim=128, seq_len=32768, dtype="bf16", rope_base=1e6, keep_first=1,
        keep_last=2, topk_chunks=30, topk_groups=48, needle_mode="pairs",
        needle_count=16, needle_shift=1.5, seed=1004),
    # the chunk-only variant (the paper's exact-token Qwen3 wrapper): 16 chunks
    # routed, every group of each opened, at the qwen32k shape
    "qwen32k_chunks": Workload(
        key="qwen32k_chunks", number=6, batch=1, n_q_heads=32, n_kv_heads=4,
        head_dim=128, seq_len=32768, dtype="bf16", rope_base=1e6, keep_first=2,
        keep_last=8, topk_chunks=16, topk_groups=64, needle_mode="pairs",
        needle_count=16, needle_shift=1.5, seed=1006),
    "decode64k": Workload(
        key="decode64k", number=5, batch=1, n_q_heads=32, n_kv_heads=4,
        head_dim=128, seq_len=65536 + 64, dtype="bf16", rope_base=1e6,
        keep_first=2, keep_last=8, topk_chunks=20, topk_groups=32,
        needle_mode="depths", needle_depths=(102, 512, 921), needle_shift=2.0,
        decode_block=True, seed=1005),
    # a context beyond 64K: 2037 routable middle chunks per unit (needles at
    # 10/50/90% depth, as in decode64k)
    "decode128k": Workload(
        key="decode128k", number=8, batch=1, n_q_heads=32, n_kv_heads=4,
        head_dim=128, seq_len=131072 + 64, dtype="bf16", rope_base=1e6,
        keep_first=2, keep_last=8, topk_chunks=20, topk_groups=32,
        needle_mode="depths", needle_depths=(204, 1024, 1843), needle_shift=2.0,
        decode_block=True, seed=1008),
    # sixteen consecutive decode blocks after the same 64K history: the
    # blocks share the needle directions (as consecutive tokens of one
    # context share what they look up), so their routing overlaps
    "decode64k_seq": Workload(
        key="decode64k_seq", number=7, batch=1, n_q_heads=32, n_kv_heads=4,
        head_dim=128, seq_len=65536 + 16 * 64, dtype="bf16", rope_base=1e6,
        keep_first=2, keep_last=8, topk_chunks=20, topk_groups=32,
        needle_mode="depths", needle_depths=(102, 512, 921), needle_shift=2.0,
        decode_block=True, decode_blocks=16, seed=1007),
}


def preset(key_or_number) -> Workload:
    if isinstance(key_or_number, int):
        for w in PRESETS.values():
            if w.number == key_or_number:
                return w
        raise KeyError(key_or_number)
    return PRESETS[key_or_number]


# ---------------------------------------------------------------- storage ---

def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64 -> fp32 (RNE) -> bf16 (RNE); returns the uint16 bit patterns."""
    f = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = f + (np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1)))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def storage_to_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of stored fp32 or bf16 (uint16 bit pattern) data."""
    if dtype == "bf16":
        return bf16_bits_to_f64(arr)
    return np.asarray(arr, dtype=np.float64)


def _to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f64_to_bf16_bits(x)
    return np.ascontiguousarray(x, dtype=np.float32)


# -------------------------------------------------------------- the model ---

def _rotary(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of x[..., t, :] at absolute positions.

    Dimension p pairs with p + d/2; the pair turns by positions * base**(-2p/d).
    """
    d = x.shape[-1]
    half = d // 2
    freq = base ** (-(np.arange(half, dtype=np.float64) * 2.0) / d)
    ang = positions.astype(np.float64)[:, None] * freq[None, :]
    cos, sin = np.cos(ang), np.sin(ang)
    lo, hi = x[..., :half], x[..., half:]
    return np.concatenate([lo * cos - hi * sin, lo * sin + hi * cos], axis=-1)


def _unit(rng: np.random.Generator, shape) -> np.ndarray:
    u = rng.standard_normal(shape)
    return u / np.linalg.norm(u, axis=-1, keepdims=True)


def _positions(w: Workload, pos: np.ndarray) -> np.ndarray:
    """RoPE positions of tokens at absolute positions ``pos``: wrapped modulo
    ``w.rope_wrap`` when set.  The wrap is a multiple of the chunk, so every
    chunk and group still holds consecutive positions."""
    if w.rope_wrap <= 0:
        return pos
    if w.rope_wrap % w.chunk:
        raise ValueError("rope_wrap must be a multiple of the chunk")
    return pos % w.rope_wrap


def generate(w: Workload, seed: int | None = None, position_offset: int = 0,
             unrounded: bool = False) -> dict:
    """Draw the inputs of workload ``w``.

    Returns a dict with storage arrays ``q`` [B, Hq, n_q_chunks*C, d] (query
    block(s) only), ``k`` and ``v`` [B, Hkv, seq_len, d] (every token of the
    sequence, history included), plus the seed and needle bookkeeping.  fp32
    presets store ``np.float32``; bf16 presets store ``np.uint16`` bit
    patterns.  ``position_offset`` shifts every absolute RoPE position (used
    to check translation invariance).  ``unrounded`` returns the float64
    values before storage rounding.
    """
    seed = w.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    B, Hq, Hkv, d, N, C = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.seq_len, w.chunk
    r = Hq // Hkv
    assert N % C == 0 and Hq % Hkv == 0
    q0_tok = w.q_chunk0 * C
    nq_tok = N - q0_tok

    q_raw = rng.standard_normal((B, Hq, nq_tok, d)) * w.prescale
    k_raw = rng.standard_normal((B, Hkv, N, d)) * w.prescale
    v = rng.standard_normal((B, Hkv, N, d))

    q = _rotary(q_raw, _positions(w, np.arange(q0_tok, N) + position_offset), w.rope_base)
    del q_raw
    k = _rotary(k_raw, _positions(w, np.arange(N) + position_offset), w.rope_base)
    del k_raw

    needles = []
    nc = w.n_chunks
    lp = max(w.keep_last, 1 if w.force_prev else 0)
    if w.needle_mode == "tail":
        # needle chunks drawn among the routable middle chunks of the last chunk
        last = nc - 1
        cand = np.arange(w.keep_first, last - lp)
        picks = rng.choice(cand, size=w.needle_count, replace=False)
        u = _unit(rng, (d,))
        for c in sorted(int(x) for x in picks):
            k[:, :, c * C:(c + 1) * C, :] += w.needle_shift * u
            needles.append((c, last))
        q[:, :, (last - w.q_chunk0) * C:, :] += w.needle_shift * u
    elif w.needle_mode == "pairs":
        lo_q = w.keep_first + lp + 1        # first query chunk with a routable middle
        for b in range(B):
            qcs = rng.choice(np.arange(lo_q, nc), size=w.needle_count, replace=False)
            ncs = [int(rng.integers(w.keep_first, int(qc) - lp)) for qc in qcs]
            dirs = _unit(rng, (w.needle_count, Hkv, d))
            for i, (qc, kc) in enumerate(zip(qcs, ncs)):
                qc = int(qc)
                for j in range(Hkv):
                    k[b, j, kc * C:(kc + 1) * C, :] += w.needle_shift * dirs[i, j]
                    q[b, j * r:(j + 1) * r, (qc - w.q_chunk0) * C:(qc - w.q_chunk0 + 1) * C, :] += \
                        w.needle_shift * dirs[i, j]
                needles.append((b, kc, qc))
    elif w.needle_mode == "depths":
        dirs = _unit(rng, (Hkv, d))
        last = nc - 1
        for kc in w.needle_depths:
            for j in range(Hkv):
                k[:, j, kc * C:(kc + 1) * C, :] += w.needle_shift * dirs[j]
            needles.append((kc, last))
        for j in range(Hkv):
            q[:, j * r:(j + 1) * r, :, :] += w.needle_shift * dirs[j]

    store = (lambda x: x) if unrounded else (lambda x: _to_storage(x, w.dtype))
    return {
        "q": store(q),
        "k": store(k),
        "v": store(v),
        "seed": seed,
        "needles": needles,
        "workload": w,
    }
