"""Routing selections on controlled summary tables, stage-isolated, through
the C ABI (Sec. 3.3: chunk scores and top-K_c, group refinement and top-K_g,
lowest index first among equal scores).

The tables and query means hold small integers (or multiples of a power of
two), so every fp32 score the kernels form is exact and equals the oracle's
float64 score: the GPU's chunk and group indices must equal the oracle's
lowest-index top-k bit for bit, ties included.  Value ranges are chosen to
make ties plentiful ("ties"), absent ("spread"), total ("zero": every score
0), or to raise the running cut of the streaming selection on every block
("ramp": scores increase with the id).

The cases reach every selection path of the routing kernels: the packed
kernel (more than 128 units; register lists up to 1024 candidates, the LDS
form of its group stage beyond), the wide kernel (at most 128 units, up to
4096 candidates: wave 0 alone below 257, the workgroup selection with one to
four keys per thread, both forms of its bound), the spread form (from q_bar,
at most 16 units with 256..4096 candidates: the table scan over several
workgroups per unit, the wide kernel's selection in the last one), the long
kernel (streaming selection beyond those lists, up to the 2^18-candidate
limit), and the separate group call."""

from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import hga_oracle as O  # noqa: E402

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


# name: (head_dim, batch, n_kv, n_q_chunks, middle chunks of the last query
#        chunk, K_c, K_g, group, values)
CASES = {
    # wide kernel (<= 128 units; from q_bar with 256..4096 candidates only
    # above 16 units, below that the spread form, whose last workgroup runs
    # the same selection)
    "wide_wave0_d128": (128, 1, 4, 1, 200, 20, 32, 16, "ties"),
    "wide_qbar_20_units": (128, 1, 4, 5, 1500, 30, 48, 16, "ties"),
    "wide_qbar_20_units_d64": (64, 1, 4, 5, 3000, 64, 96, 16, "spread"),
    "wide_per1_d128": (128, 1, 4, 1, 700, 20, 32, 16, "ties"),
    "wide_per1_zero": (128, 1, 4, 1, 700, 20, 32, 16, "zero"),
    "wide_per2_k100_g100": (128, 1, 4, 1, 1500, 100, 100, 16, "ties"),
    "wide_per2_k100_g40": (128, 1, 4, 1, 1500, 100, 40, 16, "ties"),
    "wide_per3_d128": (128, 1, 4, 1, 3000, 30, 48, 16, "spread"),
    "wide_per3_d64": (64, 2, 2, 1, 2500, 20, 32, 16, "ties"),
    "wide_per4_d64_max": (64, 1, 4, 2, 4096, 64, 64, 16, "ties"),
    "wide_g8_ng_above_256": (64, 1, 2, 3, 900, 40, 70, 8, "ties"),
    # packed kernel (> 128 units, <= 1024 candidates)
    "packed_regs16_d128": (128, 1, 2, 80, 1024, 30, 48, 16, "ties"),
    "packed_zero_d128": (128, 1, 2, 80, 1000, 30, 48, 16, "zero"),
    "packed_small_k_d64": (64, 2, 2, 40, 140, 3, 4, 16, "ties"),
    "packed_lds_groups_d64": (64, 2, 2, 40, 1000, 300, 40, 16, "ties"),
    "packed_g32_d64": (64, 1, 4, 40, 600, 12, 7, 32, "spread"),
    # long kernel (beyond the other kernels' lists)
    "long_decode_d128": (128, 1, 4, 1, 3500, 20, 32, 16, "ties"),
    "long_decode_d64": (64, 1, 4, 1, 5000, 100, 100, 16, "ties"),
    "long_ramp_d64": (64, 1, 2, 1, 20000, 64, 96, 16, "ramp"),
    "long_zero_d128": (128, 1, 2, 1, 10000, 30, 48, 16, "zero"),
    "long_many_units_d128": (128, 1, 2, 80, 1100, 30, 48, 16, "ties"),
    "long_k512_g8": (64, 1, 1, 2, 9000, 512, 512, 8, "ties"),
    "long_limit_d64": (64, 1, 1, 1, 1 << 18, 512, 512, 16, "ties"),
}


def _tables(rng, mode, B, H, T, gpc, nq, d):
    """Chunk table [B, H, T, d], group table [B, H, T*gpc, d] and q_bar
    [B, H, nq, d], float64 holding fp32-exact values."""
    if mode in ("ties", "zero"):
        cs = rng.integers(-2, 3, (B, H, T, d)).astype(np.float64)
        gs = rng.integers(-2, 3, (B, H, T * gpc, d)).astype(np.float64)
        qb = rng.integers(-2, 3, (B, H, nq, d)).astype(np.float64)
        if mode == "zero":
            qb[:] = 0.0
    elif mode == "spread":   # |score| <= d * 1000 * 50 < 2^24
        cs = rng.integers(-1000, 1001, (B, H, T, d)).astype(np.float64)
        gs = rng.integers(-1000, 1001, (B, H, T * gpc, d)).astype(np.float64)
        qb = rng.integers(-50, 51, (B, H, nq, d)).astype(np.float64)
    elif mode == "ramp":     # score of chunk m = m, of group g = g (plus small ties)
        cs = np.zeros((B, H, T, d))
        cs[..., 0] = np.arange(T)
        gs = np.zeros((B, H, T * gpc, d))
        gs[..., 0] = np.arange(T * gpc) // 2
        qb = np.zeros((B, H, nq, d))
        qb[..., 0] = 1.0
    else:
        raise ValueError(mode)
    return cs, gs, qb


def _dev(x, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dtype).cuda()


@pytest.mark.parametrize("name", list(CASES))
def test_selection_paths_match_oracle_exactly(hga, name):
    d, B, H, nq, n_last, K_c, K_g, group, mode = CASES[name]
    F, L = 1, 0
    W = 1                              # recent window with the forced previous chunk
    c_last = n_last + W + F            # middle chunks [F, c - W)
    c0 = c_last - nq + 1
    T = c_last + 1
    gpc = 64 // group
    _say(f"[select] {name}: d{d} B{B} H{H} units {B * H * nq} middle {n_last - nq + 1}..{n_last} "
         f"K_c {K_c} K_g {K_g} G{group} {mode}")
    plan = hga.Plan(batch=B, n_q_heads=H, n_kv_heads=H, head_dim=d, group=group, keep_first=F,
                    keep_last=L, force_prev=1, topk_chunks=K_c, topk_groups=K_g,
                    dtype=hga.BF16, rope_base=1e6)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    cs, gs, qb = _tables(rng, mode, B, H, T, gpc, nq, d)
    ids = list(range(c0, c0 + nq))
    want_c = O.route_chunks(qb, cs, ids, F, L, 1, K_c)
    want_g = O.route_groups(qb, want_c, gs, gpc, K_g)
    cs_t, gs_t, qb_t = _dev(cs), _dev(gs), _dev(qb)
    ci = torch.full((B, H, nq, K_c), -7, dtype=torch.int32, device="cuda")
    gi = torch.full((B, H, nq, K_g), -7, dtype=torch.int32, device="cuda")
    hga.hga_route_qbar(plan, qb_t, c0, cs_t, gs_t, ci, gi)
    torch.cuda.synchronize()
    got_c, got_g = ci.cpu().numpy(), gi.cpu().numpy()
    bad = np.argwhere(np.any(got_c != want_c, axis=-1))
    assert bad.size == 0, f"chunk_idx differs at {bad[:3].tolist()}: {got_c[tuple(bad[0])]} vs " \
                          f"{want_c[tuple(bad[0])]}"
    bad = np.argwhere(np.any(got_g != want_g, axis=-1))
    assert bad.size == 0, f"group_idx differs at {bad[:3].tolist()}: {got_g[tuple(bad[0])]} vs " \
                          f"{want_g[tuple(bad[0])]}"
    # the separate group call on the same chunk selection
    gi2 = torch.full_like(gi, -7)
    hga.hga_route_groups(plan, qb_t, ci, c0, gs_t, gi2)
    torch.cuda.synchronize()
    assert np.array_equal(gi2.cpu().numpy(), want_g)
    n_tied = 0
    for b in range(B):
        for j in range(H):
            M = np.arange(F, c_last - W)
            sc = cs[b, j, M] @ qb[b, j, -1]
            k = min(K_c, M.size)
            kth = np.sort(sc)[::-1][k - 1]
            n_tied += int(np.sum(sc == kth) > 1)
    _say(f"  exact; selections with a tie at the cut (last query chunk): {n_tied} of {B * H}")


@pytest.mark.parametrize("name,r", [("packed_regs16_d128", 2), ("wide_per1_d128", 8),
                                    ("long_decode_d128", 8), ("long_many_units_d128", 2)])
def test_selection_from_query_rows(hga, name, r):
    """hga_route and hga_route_chunks forming q_bar from integer query rows
    (the mean over r*64 rows, a power of two, is exact): q_bar, chunk and
    group indices equal the oracle's bit for bit."""
    d, B, H, nq, n_last, K_c, K_g, group, mode = CASES[name]
    F, L, W = 1, 0, 1
    c_last = n_last + W + F
    c0 = c_last - nq + 1
    T = c_last + 1
    gpc = 64 // group
    _say(f"[select from q] {name} r{r}")
    plan = hga.Plan(batch=B, n_q_heads=H * r, n_kv_heads=H, head_dim=d, group=group,
                    keep_first=F, keep_last=L, force_prev=1, topk_chunks=K_c, topk_groups=K_g,
                    dtype=hga.BF16, rope_base=1e6)
    rng = np.random.default_rng(99)
    cs, gs, _ = _tables(rng, "ties", B, H, T, gpc, nq, d)
    q = rng.integers(-3, 4, (B, H * r, nq * 64, d)).astype(np.float64)
    qb = O.query_means(q, H, 64)
    ids = list(range(c0, c0 + nq))
    want_c = O.route_chunks(qb, cs, ids, F, L, 1, K_c)
    want_g = O.route_groups(qb, want_c, gs, gpc, K_g)
    q_t = _dev(q, torch.bfloat16)
    cs_t, gs_t = _dev(cs), _dev(gs)
    for fused in (True, False):
        qbar = torch.full((B, H, nq, d), float("nan"), device="cuda")
        ci = torch.full((B, H, nq, K_c), -7, dtype=torch.int32, device="cuda")
        gi = torch.full((B, H, nq, K_g), -7, dtype=torch.int32, device="cuda")
        if fused:
            hga.hga_route(plan, q_t, c0, cs_t, gs_t, qbar, ci, gi)
        else:
            hga.hga_route_chunks(plan, q_t, c0, cs_t, qbar, ci)
            hga.hga_route_groups(plan, qbar, ci, c0, gs_t, gi)
        torch.cuda.synchronize()
        assert np.array_equal(qbar.cpu().numpy().astype(np.float64), qb)
        assert np.array_equal(ci.cpu().numpy(), want_c)
        assert np.array_equal(gi.cpu().numpy(), want_g)


def test_candidate_limit_refused_before_launch(hga):
    """One middle chunk beyond 2^18 is refused (HGA_EUNSUPPORTED) before any
    launch; the outputs stay untouched."""
    F, W = 1, 1
    n = (1 << 18) + 1
    c = n + W + F
    plan = hga.Plan(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64, topk_chunks=8,
                    topk_groups=8, dtype=hga.BF16, rope_base=1e6)
    cs = torch.zeros(1, 1, c + 1, 64, device="cuda")
    gs = torch.zeros(1, 1, (c + 1) * 4, 64, device="cuda")
    qb = torch.zeros(1, 1, 1, 64, device="cuda")
    ci = torch.full((1, 1, 1, 8), -7, dtype=torch.int32, device="cuda")
    gi = torch.full((1, 1, 1, 8), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(hga.HgaError) as e:
        hga.hga_route_qbar(plan, qb, c, cs, gs, ci, gi)
    assert e.value.status == -2
    torch.cuda.synchronize()
    assert bool((ci == -7).all()) and bool((gi == -7).all())


def test_spread_route_reuses_the_plan_workspace(hga):
    """hga_route_qbar's spread form (at most 16 units, 256..4096 candidates)
    meets each unit's keys in the plan's workspace and leaves its counters at
    zero: successive calls on one plan, with different unit and candidate
    counts and inputs, each equal the oracle's lowest-index top-k exactly."""
    d, B, H, K_c, K_g, group = 128, 1, 4, 20, 32, 16
    F, L, W = 1, 0, 1
    gpc = 64 // group
    plan = hga.Plan(batch=B, n_q_heads=H, n_kv_heads=H, head_dim=d, group=group, keep_first=F,
                    keep_last=L, force_prev=1, topk_chunks=K_c, topk_groups=K_g,
                    dtype=hga.BF16, rope_base=1e6)
    for call, (nq, n_last, mode) in enumerate([(1, 700, "ties"), (4, 3000, "spread"),
                                                (2, 300, "ties"), (1, 4000, "zero"),
                                                (3, 1500, "ramp")]):
        c_last = n_last + W + F
        c0 = c_last - nq + 1
        T = c_last + 1
        _say(f"[spread reuse] call {call}: units {B * H * nq} middle {n_last} {mode}")
        rng = np.random.default_rng(1000 + call)
        cs, gs, qb = _tables(rng, mode, B, H, T, gpc, nq, d)
        ids = list(range(c0, c0 + nq))
        want_c = O.route_chunks(qb, cs, ids, F, L, 1, K_c)
        want_g = O.route_groups(qb, want_c, gs, gpc, K_g)
        ci = torch.full((B, H, nq, K_c), -7, dtype=torch.int32, device="cuda")
        gi = torch.full((B, H, nq, K_g), -7, dtype=torch.int32, device="cuda")
        hga.hga_route_qbar(plan, _dev(qb), c0, _dev(cs), _dev(gs), ci, gi)
        torch.cuda.synchronize()
        assert np.array_equal(ci.cpu().numpy(), want_c), f"call {call}: chunk_idx"
        assert np.array_equal(gi.cpu().numpy(), want_g), f"call {call}: group_idx"
