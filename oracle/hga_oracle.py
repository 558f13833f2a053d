"""Plain float64 NumPy oracle of HGA's routed-attention path.

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the benchmark's
CPU-baseline leg, never by the product path.  It shares no code with the HIP
library; the only thing both sides consume is the seeded input generator.

Paper: "Hierarchical Global Attention: Drop-In Exact-Token Routing for
Pretrained Long-Context Transformers".  Every function follows one passage
and computes it in float64, step by step in the paper's order, with no
blocking or fusion beyond what the definition states.

Readings of points the paper leaves open (each is also listed in the design
notes of the repository):

* RoPE is rotate-half: dimension p pairs with p + d/2, the pair turns by
  theta_p = base**(-2p/d) per position (Sec. 2 "RoPE"; the Qwen3 layout the
  wrapper keeps, Sec. 4.1).
* A pair is "high-frequency" for a span when its wavelength 2*pi/theta_p is
  at most the span (Sec. 3.2 gives no threshold).
* The "middle position" of a span is its real-valued centre,
  start + (span - 1) / 2 (Sec. 3.2).
* Summaries are means (Sec. 3.2 allows sums or means; every summarised span
  is full, so the ranking is identical).
* The query side of chunk routing is the mean of the rotated queries over the
  chunk's tokens and over the query heads sharing the KV head (chunk-shared
  routing, Sec. 1; per-KV-head routing, Sec. 3.3).  Scores are unscaled dot
  products.
* Ties are broken by the lowest index; selections are emitted ascending and
  padded with -1.  With fewer candidates than the budget, all are taken.
* Group refinement selects the top groups globally across the selected
  chunks (Sec. 3.3).
* The recent window always contains the preceding chunk: with L recent
  chunks and the force-include rule, the window is max(L, 1) chunks
  (Sec. 3.3 "Deterministic visibility").
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "rope_inv_freq", "high_freq_pairs", "rotate_pairs", "span_phases",
    "summaries", "summaries_literal", "summary_magnitudes",
    "query_means", "query_magnitudes", "visibility", "topk_lowest_index",
    "route_chunks", "route_groups", "gather", "working_set", "attend",
    "hga_forward", "fetched_tokens",
]


# ------------------------------------------------------------------ RoPE ---

def rope_inv_freq(head_dim: int, base: float) -> np.ndarray:
    """theta_p = base**(-2p/d) for pairs p = 0 .. d/2-1 (Sec. 2 "RoPE")."""
    p = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * p / head_dim)


def high_freq_pairs(span: int, head_dim: int, base: float) -> int:
    """Number of high-frequency pairs for a span (Sec. 3.2; reading: wavelength <= span)."""
    theta = rope_inv_freq(head_dim, base)
    return int(np.count_nonzero(2.0 * math.pi / theta <= span))


def rotate_pairs(x: np.ndarray, angle: np.ndarray) -> np.ndarray:
    """Apply R(angle) to every rotate-half pair of x[..., d].

    ``angle`` broadcasts against x[..., :d/2].  R(phi)(a, b) =
    (a cos phi - b sin phi, a sin phi + b cos phi).
    """
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    c, s = np.cos(angle), np.sin(angle)
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


# ------------------------------------------------------------- summaries ---

def span_phases(span: int, head_dim: int, base: float, n_hf: int) -> np.ndarray:
    """phi_p(o) for offsets o in [0, span): the angle that takes a key rotated
    at (start + o) to the rotation it would have at the span's middle position.

    High-frequency pairs (p < n_hf) keep their own rotation (phi = 0);
    low-frequency pairs get ((span - 1)/2 - o) * theta_p.  Shape [span, d/2].
    """
    theta = rope_inv_freq(head_dim, base)
    o = np.arange(span, dtype=np.float64)
    phi = ((span - 1) / 2.0 - o)[:, None] * theta[None, :]
    phi[:, :n_hf] = 0.0
    return phi


def summaries(k_rot: np.ndarray, span: int, base: float, n_hf: int) -> np.ndarray:
    """Mixed-RoPE key summaries of every full span (Sec. 3.2).

    k_rot: [B, H, N, d] keys already rotated at their absolute positions.
    Returns [B, H, N // span, d]: the mean over the span's tokens of
    R(phi_p(o)) k_rot.  For a high-frequency pair this is the mean of the
    rotated keys; for a low-frequency pair it equals the mean of the raw keys
    rotated at the middle position (the identity is checked against
    ``summaries_literal``).
    """
    B, H, N, d = k_rot.shape
    n = N // span
    kk = np.asarray(k_rot[:, :, :n * span, :], dtype=np.float64).reshape(B, H, n, span, d)
    phi = span_phases(span, d, base, n_hf)          # [span, d/2]
    return rotate_pairs(kk, phi[:, :]).mean(axis=3)


def summaries_literal(k_rot: np.ndarray, span: int, base: float, n_hf: int,
                      first_position: int = 0, wrap: int = 0) -> np.ndarray:
    """The paper's two-part rule taken literally (Sec. 3.2).

    Keys are un-rotated to raw space with their RoPE positions
    (first_position + t, taken modulo ``wrap`` when it is set: the variant of
    Sec. 5 on long-context positional encoding).  High-frequency pairs:
    rotate per token (that is, keep k_rot) and average.  Low-frequency pairs:
    average the raw keys, then rotate the average at the span's middle
    position, the mean of its tokens' positions.
    """
    B, H, N, d = k_rot.shape
    half = d // 2
    n = N // span
    theta = rope_inv_freq(d, base)
    pos = first_position + np.arange(n * span, dtype=np.float64)
    if wrap:
        pos = np.mod(pos, wrap)
    k = np.asarray(k_rot[:, :, :n * span, :], dtype=np.float64)
    raw = rotate_pairs(k, -pos[:, None] * theta[None, :])
    rot_mean = k.reshape(B, H, n, span, d).mean(axis=3)
    raw_mean = raw.reshape(B, H, n, span, d).mean(axis=3)
    middle = pos.reshape(n, span).mean(axis=1)
    low = rotate_pairs(raw_mean, middle[:, None] * theta[None, :])
    out = low.copy()
    out[..., :n_hf] = rot_mean[..., :n_hf]
    out[..., half:half + n_hf] = rot_mean[..., half:half + n_hf]
    return out


def summary_magnitudes(k_rot: np.ndarray, span: int, base: float, n_hf: int) -> np.ndarray:
    """Mean over the span of |a cos phi| + |b sin phi| (first half) and
    |a sin phi| + |b cos phi| (second half): the magnitude each summary
    element is accumulated from.  Used only to bound the rounding error of a
    single-precision evaluation when comparing selections."""
    B, H, N, d = k_rot.shape
    half = d // 2
    n = N // span
    kk = np.asarray(k_rot[:, :, :n * span, :], dtype=np.float64).reshape(B, H, n, span, d)
    phi = span_phases(span, d, base, n_hf)
    a, b = np.abs(kk[..., :half]), np.abs(kk[..., half:])
    c, s = np.abs(np.cos(phi)), np.abs(np.sin(phi))
    return np.concatenate([a * c + b * s, a * s + b * c], axis=-1).mean(axis=3)


# --------------------------------------------------------------- queries ---

def query_means(q_rot: np.ndarray, n_kv_heads: int, chunk: int) -> np.ndarray:
    """q_bar[b, j, c]: mean of the rotated queries over the chunk's tokens and
    over the query heads that share KV head j (GQA, Sec. 2; chunk-shared
    routing, Sec. 1 and Sec. 3.3).  q_rot: [B, Hq, n*chunk, d] ->
    [B, Hkv, n, d]."""
    B, Hq, T, d = q_rot.shape
    r = Hq // n_kv_heads
    qq = np.asarray(q_rot, dtype=np.float64).reshape(B, n_kv_heads, r, T // chunk, chunk, d)
    return qq.mean(axis=(2, 4))


def query_magnitudes(q_rot: np.ndarray, n_kv_heads: int, chunk: int) -> np.ndarray:
    """Mean of |q_rot| over the same tokens and heads as ``query_means``."""
    return query_means(np.abs(np.asarray(q_rot, dtype=np.float64)), n_kv_heads, chunk)


# ----------------------------------------------------------- visibility ---

def visibility(c: int, keep_first: int, keep_last: int, force_prev: int = 1):
    """Deterministic and routable chunks for query chunk c (Sec. 3.3).

    Returns (D, M): D = the always-visible closed chunks (the first
    ``keep_first`` sink chunks and the recent window, which always contains
    chunk c-1 when force-include is on), ascending; M = the middle chunks
    that compete for the route budget, ascending.  The current chunk c is
    visible as well, under a causal mask; it is in neither list.
    """
    window = max(keep_last, 1 if force_prev else 0)
    first = set(range(0, min(keep_first, c)))
    recent = set(range(max(0, c - window), c))
    D = sorted(first | recent)
    M = list(range(keep_first, c - window)) if c - window > keep_first else []
    return D, M


def topk_lowest_index(scores: np.ndarray, ids: np.ndarray, k: int) -> np.ndarray:
    """The k ids with the largest scores, lowest id first among equal
    scores; returned in ascending id order."""
    order = np.lexsort((ids, -scores))
    return np.sort(ids[order[:k]])


# --------------------------------------------------------------- routing ---

def route_chunks(qbar: np.ndarray, chunk_sum: np.ndarray, q_chunk_ids, keep_first: int,
                 keep_last: int, force_prev: int, topk: int, details: bool = False):
    """Chunk-level content routing (Sec. 3.3 "Content-based middle routing").

    qbar: [B, Hkv, nq, d] for the query chunks ``q_chunk_ids`` (absolute).
    chunk_sum: [B, Hkv, n_table, d].  For each (b, j, c) the middle chunks M_c
    are scored by q_bar . chunk_sum and the top min(topk, |M_c|) kept.
    Returns chunk_idx [B, Hkv, nq, topk] int32 (ascending, -1 padded) and, if
    ``details``, a list of (b, j, i, candidate ids, scores) per selection.
    """
    B, H, nq, d = qbar.shape
    out = np.full((B, H, nq, topk), -1, dtype=np.int32)
    info = []
    for i, c in enumerate(q_chunk_ids):
        _, M = visibility(int(c), keep_first, keep_last, force_prev)
        if not M:
            continue
        M = np.asarray(M, dtype=np.int64)
        scores = np.einsum("bhd,bhmd->bhm", qbar[:, :, i], chunk_sum[:, :, M])
        k = min(topk, len(M))
        for b in range(B):
            for j in range(H):
                out[b, j, i, :k] = topk_lowest_index(scores[b, j], M, k)
                if details:
                    info.append((b, j, i, M, scores[b, j]))
    return (out, info) if details else out


def route_groups(qbar: np.ndarray, chunk_idx: np.ndarray, group_sum: np.ndarray,
                 groups_per_chunk: int, topk: int, details: bool = False):
    """Group refinement inside the selected chunks (Sec. 3.3).

    The candidates are every group of every selected chunk (global group id
    groups_per_chunk * c' + i); they are scored by q_bar . group_sum and the
    top min(topk, #candidates) are opened, globally across the chunks.
    Returns group_idx [B, Hkv, nq, topk] int32 (ascending, -1 padded).
    """
    B, H, nq, _ = qbar.shape
    out = np.full((B, H, nq, topk), -1, dtype=np.int32)
    info = []
    for b in range(B):
        for j in range(H):
            for i in range(nq):
                chunks = chunk_idx[b, j, i]
                chunks = chunks[chunks >= 0].astype(np.int64)
                if chunks.size == 0:
                    continue
                cand = (chunks[:, None] * groups_per_chunk
                        + np.arange(groups_per_chunk)[None, :]).reshape(-1)
                scores = group_sum[b, j, cand] @ qbar[b, j, i]
                k = min(topk, cand.size)
                out[b, j, i, :k] = topk_lowest_index(scores, cand, k)
                if details:
                    info.append((b, j, i, cand, scores))
    return (out, info) if details else out


# ---------------------------------------------------------------- gather ---

def gather(group_idx: np.ndarray, k: np.ndarray, v: np.ndarray, group: int):
    """Store operation "gather exact token K/V" (Sec. 4.3): slot s of query
    chunk i receives the ``group`` tokens of group group_idx[..., i, s];
    padded slots (-1) are zero.  k, v: [B, Hkv, N, d] ->
    [B, Hkv, nq, topk * group, d] each."""
    B, H, nq, kg = group_idx.shape
    d = k.shape[-1]
    ko = np.zeros((B, H, nq, kg * group, d), dtype=k.dtype)
    vo = np.zeros_like(ko)
    for b in range(B):
        for j in range(H):
            for i in range(nq):
                for s, g in enumerate(group_idx[b, j, i]):
                    if g < 0:
                        continue
                    ko[b, j, i, s * group:(s + 1) * group] = k[b, j, g * group:(g + 1) * group]
                    vo[b, j, i, s * group:(s + 1) * group] = v[b, j, g * group:(g + 1) * group]
    return ko, vo


# ------------------------------------------------------------- attention ---

def working_set(c: int, groups, chunk: int, group: int, keep_first: int,
                keep_last: int, force_prev: int) -> np.ndarray:
    """Token positions of the closed-history working set of query chunk c
    (Sec. 3.4 items 2 and 3): the always-visible first and recent chunks and
    the opened groups.  The current chunk (item 1) is added under a causal
    mask by ``attend``."""
    D, _ = visibility(c, keep_first, keep_last, force_prev)
    parts = [np.arange(cc * chunk, (cc + 1) * chunk) for cc in D]
    parts += [np.arange(int(g) * group, (int(g) + 1) * group) for g in groups if g >= 0]
    if not parts:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(parts).astype(np.int64)


def attend(q_rot: np.ndarray, k_rot: np.ndarray, v: np.ndarray, group_idx: np.ndarray,
           q_chunk_ids, chunk: int, group: int, keep_first: int, keep_last: int,
           force_prev: int, units=None):
    """Exact-token output attention (Sec. 3.4) with the causal softmax of Eq. (1).

    q_rot: [B, Hq, nq*chunk, d] queries of the chunks ``q_chunk_ids``;
    k_rot, v: [B, Hkv, N, d] for every token of the sequence (absolute
    positions); group_idx: [B, Hkv, nq, K_g].  For query head h (KV head
    h // r) and token t of chunk c, the softmax of q.k/sqrt(d) runs over the
    working set of c plus the current-chunk tokens u <= t.
    Returns (out [B, Hq, nq*chunk, d], lse [B, Hq, nq*chunk]), natural-log
    LSE.  ``units``, if given, is an iterable of (b, j, i) to evaluate; the
    other rows are left NaN.
    """
    B, Hq, T, d = q_rot.shape
    Hkv = k_rot.shape[1]
    r = Hq // Hkv
    out = np.full((B, Hq, T, d), np.nan)
    lse = np.full((B, Hq, T), np.nan)
    scale = 1.0 / math.sqrt(d)
    if units is None:
        units = [(b, j, i) for b in range(B) for j in range(Hkv) for i in range(len(q_chunk_ids))]
    causal = np.tril(np.ones((chunk, chunk), dtype=bool))   # [query t, key u]: u <= t
    for (b, j, i) in units:
        c = int(q_chunk_ids[i])
        hist = working_set(c, group_idx[b, j, i], chunk, group, keep_first, keep_last, force_prev)
        cur = np.arange(c * chunk, (c + 1) * chunk)
        keys = np.asarray(k_rot[b, j, np.concatenate([hist, cur])], dtype=np.float64)
        vals = np.asarray(v[b, j, np.concatenate([hist, cur])], dtype=np.float64)
        qs = np.asarray(q_rot[b, j * r:(j + 1) * r, i * chunk:(i + 1) * chunk], dtype=np.float64)
        logits = (qs @ keys.T) * scale                     # [r, chunk, |hist| + chunk]
        cur_part = logits[:, :, hist.size:]
        cur_part[:, ~causal] = -np.inf
        m = logits.max(axis=-1, keepdims=True)
        p = np.exp(logits - m)
        den = p.sum(axis=-1, keepdims=True)
        out[b, j * r:(j + 1) * r, i * chunk:(i + 1) * chunk] = (p @ vals) / den
        lse[b, j * r:(j + 1) * r, i * chunk:(i + 1) * chunk] = (m + np.log(den))[..., 0]
    return out, lse


def attend_backward(q_rot: np.ndarray, k_rot: np.ndarray, v: np.ndarray, dout: np.ndarray,
                    group_idx: np.ndarray, q_chunk_ids, chunk: int, group: int,
                    keep_first: int, keep_last: int, force_prev: int, units=None):
    """Gradients of the exact-token attention of ``attend`` (Sec. 3.4,
    Eq. (1)) with respect to its inputs, for the output gradient ``dout``
    [B, Hq, nq*chunk, d].  Routing is not differentiated (the selected sets
    are fixed); the routed rows are the resident rows they were gathered
    from, so their gradients land on those token rows.

    For query row i of a unit with working set X (visible chunks, opened
    groups, current-chunk tokens u <= t) and logits s_ix = q_i.k_x / sqrt(d),
    p_ix = softmax_x(s_ix), o_i = sum_x p_ix v_x, the chain rule gives
        dv_x += sum_i p_ix dout_i,
        dp_ix = dout_i . v_x,   D_i = sum_x p_ix dp_ix = dout_i . o_i,
        ds_ix = p_ix (dp_ix - D_i),
        dq_i = sum_x ds_ix k_x / sqrt(d),   dk_x += sum_i ds_ix q_i / sqrt(d).
    Returns (dq like q_rot, dk and dv like k_rot), float64; rows of query
    units not listed in ``units`` get no contribution (dq stays zero there).
    """
    B, Hq, T, d = q_rot.shape
    Hkv = k_rot.shape[1]
    r = Hq // Hkv
    dq = np.zeros((B, Hq, T, d))
    dk = np.zeros(k_rot.shape)
    dv = np.zeros(v.shape)
    scale = 1.0 / math.sqrt(d)
    if units is None:
        units = [(b, j, i) for b in range(B) for j in range(Hkv) for i in range(len(q_chunk_ids))]
    causal = np.tril(np.ones((chunk, chunk), dtype=bool))
    for (b, j, i) in units:
        c = int(q_chunk_ids[i])
        hist = working_set(c, group_idx[b, j, i], chunk, group, keep_first, keep_last, force_prev)
        cur = np.arange(c * chunk, (c + 1) * chunk)
        idx = np.concatenate([hist, cur])
        keys = np.asarray(k_rot[b, j, idx], dtype=np.float64)          # [X, d]
        vals = np.asarray(v[b, j, idx], dtype=np.float64)
        rows = slice(i * chunk, (i + 1) * chunk)
        qs = np.asarray(q_rot[b, j * r:(j + 1) * r, rows], dtype=np.float64)   # [r, C, d]
        go = np.asarray(dout[b, j * r:(j + 1) * r, rows], dtype=np.float64)
        logits = (qs @ keys.T) * scale                                  # [r, C, X]
        logits[:, :, hist.size:][:, ~causal] = -np.inf
        p = np.exp(logits - logits.max(axis=-1, keepdims=True))
        p /= p.sum(axis=-1, keepdims=True)
        dp = go @ vals.T                                                # [r, C, X]
        big_d = (p * dp).sum(axis=-1, keepdims=True)
        ds = p * (dp - big_d)
        dq[b, j * r:(j + 1) * r, rows] = (ds @ keys) * scale
        np.add.at(dk[b, j], idx, np.einsum("hcx,hcd->xd", ds, qs) * scale)
        np.add.at(dv[b, j], idx, np.einsum("hcx,hcd->xd", p, go))
    return dq, dk, dv


def fetched_tokens(c: int, n_groups: int, chunk: int, group: int, keep_first: int,
                   keep_last: int, force_prev: int) -> int:
    """Size of the closed-history working set of chunk c with n_groups opened
    groups (the tokens fetched for the block, Sec. 3.6)."""
    return int(working_set(c, list(range(n_groups)), chunk, group, keep_first,
                           keep_last, force_prev).size)


# ------------------------------------------------------------- pipeline ---

def hga_forward(q_rot, k_rot, v, *, chunk, group, keep_first, keep_last, force_prev,
                topk_chunks, topk_groups, rope_base, q_chunk0=0, n_hf_chunk=None,
                n_hf_group=None, attend_units=None, with_gather=False):
    """All five steps for the query chunks starting at ``q_chunk0``.

    q_rot: [B, Hq, nq*chunk, d]; k_rot, v: [B, Hkv, N, d] float64 (every
    token up to and including the last query chunk).  Summaries are built for
    every chunk of k_rot.
    """
    B, Hq, T, d = q_rot.shape
    Hkv = k_rot.shape[1]
    nq = T // chunk
    if n_hf_chunk is None:
        n_hf_chunk = high_freq_pairs(chunk, d, rope_base)
    if n_hf_group is None:
        n_hf_group = high_freq_pairs(group, d, rope_base)
    ids = list(range(q_chunk0, q_chunk0 + nq))
    res = {}
    res["chunk_sum"] = summaries(k_rot, chunk, rope_base, n_hf_chunk)
    res["group_sum"] = summaries(k_rot, group, rope_base, n_hf_group)
    res["qbar"] = query_means(q_rot, Hkv, chunk)
    res["chunk_idx"] = route_chunks(res["qbar"], res["chunk_sum"], ids, keep_first,
                                    keep_last, force_prev, topk_chunks)
    res["group_idx"] = route_groups(res["qbar"], res["chunk_idx"], res["group_sum"],
                                    chunk // group, topk_groups)
    if with_gather:
        res["k_routed"], res["v_routed"] = gather(res["group_idx"], k_rot, v, group)
    res["out"], res["lse"] = attend(q_rot, k_rot, v, res["group_idx"], ids, chunk, group,
                                    keep_first, keep_last, force_prev, units=attend_units)
    return res
