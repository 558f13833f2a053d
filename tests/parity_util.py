"""Comparison helpers for GPU-vs-oracle parity (test infrastructure)."""

from __future__ import annotations

import numpy as np

from oracle import hga_oracle as O
from paper_2606_30709_amd import workloads as W

U32 = 2.0 ** -24  # unit roundoff of fp32

# Output tolerances: max-abs for the attention output (bf16 / fp32 paths) and
# for the natural-log LSE (fp32 accumulators in both paths; the bf16 path's
# logits carry the fp32 error of a 64/128-term bf16 dot product).
OUT_TOL = {"f32": 1e-5, "bf16": 2e-2}
LSE_TOL = {"f32": 1e-4, "bf16": 2e-3}
# Attention backward (bf16 inputs): the weights P and dS enter the matrix
# products rounded to bf16 (unit roundoff 2^-9), so every term of the
# gradient sums carries a relative error up to 2^-9 and the normwise error of
# dq, dk, dv is about 2^-9 (measured 1.6-1.8e-3).  Bar: normwise error <=
# 2 * 2^-9 = BWD_TOL / 4 and every element within BWD_TOL = 2^-6 of the
# gradient's largest magnitude.
BWD_TOL = 2.0 ** -6


def f64(x, dtype):
    return W.storage_to_f64(x, dtype)


def tensor_to_f64(t):
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return W.bf16_bits_to_f64(t.view(torch.int16).numpy().view(np.uint16))
    return t.to(torch.float64).numpy()


def summary_bound(mag, span):
    """Forward-error bound of an fp32 span-mean evaluated from fp32 phase
    factors: span accumulations of two-product terms, table rounding."""
    return 2.0 * (span + 8) * U32 * mag


def score_bounds(qbar, summ, qmag, smag, span, rC, d):
    """Per-candidate bound on |fp32 score - exact score| (rows of summ)."""
    aq, asum = np.abs(qbar), np.abs(summ)
    return 2.0 * U32 * ((span + 8) * (smag @ aq) + (rC + 8) * (asum @ qmag)
                        + (d + 8) * (asum @ aq))


class SelectionReport:
    def __init__(self):
        self.exact = 0

    def __repr__(self):
        return f"SelectionReport(exact={self.exact})"


def check_selection(gpu_row, cand, scores, eps, k_budget, report, where=""):
    """The GPU's selection must be the oracle's top-k (ties -> lowest id),
    bit for bit.  On a difference the failure names the oracle's margin at the
    cut (k-th minus (k+1)-th score) and the fp32 error bounds of the two sides
    of the cut, so a near-tie (margin within the bounds: a rounding-order
    ambiguity of the fp32 evaluation) can be told from a wrong selection."""
    k = min(k_budget, len(cand))
    gpu = [int(x) for x in gpu_row]
    valid = [x for x in gpu if x >= 0]
    assert gpu[len(valid):] == [-1] * (len(gpu) - len(valid)), f"{where}: padding not at end {gpu}"
    assert len(valid) == k, f"{where}: selected {len(valid)} of {k}: {gpu}"
    assert valid == sorted(set(valid)), f"{where}: not ascending/distinct {gpu}"
    cand = np.asarray(cand)
    pos = {int(c): n for n, c in enumerate(cand)}
    assert all(x in pos for x in valid), f"{where}: selected a non-candidate {gpu}"
    want = list(O.topk_lowest_index(np.asarray(scores), cand, k))
    if valid == want:
        report.exact += 1
        return
    scores = np.asarray(scores)
    order = np.lexsort((cand, -scores))
    kth, nxt = order[k - 1], order[k] if k < len(cand) else order[k - 1]
    margin = float(scores[kth] - scores[nxt])
    bound = float(eps[kth] + eps[nxt])
    kind = "near-tie (margin within the fp32 bounds)" if margin <= 2 * bound else "wrong selection"
    raise AssertionError(f"{where}: {kind}: gpu {valid} oracle {want}; margin {margin:.3g}, "
                         f"bounds {float(eps[kth]):.3g} + {float(eps[nxt]):.3g}")
