"""Decode cache (App. B "Decode cache") and reserved capacity, through the ABI.

* pisa_pyramid_append from n_old to N equals pisa_build_pyramid at N bit for
  bit (same arithmetic by construction) and the float64 oracle within the
  pyramid tolerance, across new blocks, block boundaries, level growth,
  ragged tails and a rebuild from nothing (n_old = 0).
* A problem whose k, v and pyramid reserve Ncap > N rows (the rows past N
  filled with large junk) gives the same indices, outputs and lse as the same
  problem laid out compactly, for every selection schedule and attention path.
* A short streaming decode loop (append one token, select, attend) matches
  the oracle step by step.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import dev

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None

JUNK = 1.0e4  # value of the reserved rows past N: any read of them shows up


def _reserved(x: np.ndarray, cap: int, dtype: str) -> torch.Tensor:
    """[B, Hkv, N, d] -> device [B, Hkv, cap, d] with junk rows past N."""
    B, Hkv, N, d = x.shape
    full = np.full((B, Hkv, cap, d), JUNK, dtype=np.float32)
    full[:, :, :N] = x
    return dev(full, dtype)


def _valid_rows(p):
    """(first row, rows) of every stored level of problem p."""
    offs, _ = pisa.pisa_pyramid_layout(p)
    sizes = O.level_sizes(p.N, p.C, p.fanout)
    nst = max(1, len(sizes) - 1)
    return [(offs[l], sizes[l]) for l in range(nst)]


APPEND = [
    # (dtype, Hkv, d, C, g, n_old, N, cap)
    ("bf16", 2, 128, 64, 2, 1000, 1001, 4096),
    ("bf16", 2, 128, 64, 2, 1023, 1024, 4096),
    ("bf16", 2, 128, 64, 2, 1024, 1025, 4096),
    ("bf16", 2, 128, 64, 2, 1024, 2049, 4096),
    ("bf16", 2, 128, 64, 2, 0, 777, 1024),
    ("bf16", 1, 128, 64, 2, 1, 5000, 5000),
    ("f32", 2, 64, 32, 3, 700, 1950, 2000),
    ("bf16", 2, 128, 128, 4, 3000, 9000, 9000),
    # one token into the last block (the per-token decode path)
    ("f32", 2, 64, 32, 3, 1949, 1950, 2000),
    ("bf16", 2, 128, 128, 4, 8999, 9000, 9000),
    ("bf16", 1, 64, 32, 2, 4095, 4096, 8192),
]


@pytest.mark.parametrize("case", APPEND, ids=[f"{c[0]}-C{c[3]}-g{c[4]}-{c[5]}to{c[6]}" for c in APPEND])
def test_append_equals_full_build(case):
    dtype, Hkv, d, C, g, n_old, N, cap = case
    print(f"[decode-cache] append {case}", flush=True)
    r = np.random.default_rng(n_old * 31 + N)
    k = r.standard_normal((1, Hkv, N, d), dtype=np.float32)
    if dtype == "bf16":
        k = inputs.round_to_bf16(k)
    kd = _reserved(k, cap, dtype)
    p_new = pisa.make_problem(1, Hkv, Hkv, 1, N, d, C, g, 4, 1, dtype, Ncap=cap)
    _, R = pisa.pisa_pyramid_layout(p_new)
    pyr = torch.zeros((1, Hkv, R, d), dtype=torch.float32, device="cuda")
    if n_old > 0:
        p_old = pisa.make_problem(1, Hkv, Hkv, 1, n_old, d, C, g, 4, 1, dtype, Ncap=cap)
        pisa.pisa_build_pyramid(p_old, kd, pyr)
    pisa.pisa_pyramid_append(p_new, kd, pyr, n_old)
    full = torch.full((1, Hkv, R, d), float("nan"), dtype=torch.float32, device="cuda")
    pisa.pisa_build_pyramid(p_new, kd, full)
    torch.cuda.synchronize()
    want = O.pyramid(k, C, g)
    L = len(O.level_sizes(N, C, g))
    tol = (C + L * g) * 2.0 ** -24 * float(np.abs(k).max())
    row = 0
    for first, n in _valid_rows(p_new):
        a, b = pyr[:, :, first:first + n], full[:, :, first:first + n]
        assert torch.equal(a, b), (first, n)
        err = np.abs(a.cpu().numpy() - want[:, :, row:row + n]).max()
        assert err <= tol, (first, err)
        row += n


def _run_all(p, q, k, v, schedule):
    p.schedule = schedule
    pyr = pisa.build_pyramid(p, k)
    idx, sc = pisa.select(p, q, k, pyr, with_score=True)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    bsa = pisa.select_flat_bsa(p, q, pyr) if schedule == pisa.PISA_SCHEDULE_AUTO else None
    torch.cuda.synchronize()
    return idx, sc, o, lse, bsa


CAPACITY = [
    # (name, B, H, Hkv, Nq, N, d, C, g, K, causal, dtype, extra rows)
    ("prefill-bf16", 1, 4, 2, 3000, 3000, 128, 64, 2, 8, 1, "bf16", 300),
    ("decode-bf16", 2, 4, 2, 1, 5000, 128, 64, 2, 8, 1, "bf16", 1000),
    ("mid-f32", 1, 2, 2, 500, 2500, 64, 32, 3, 5, 0, "f32", 77),
]


@pytest.mark.parametrize("case", CAPACITY, ids=[c[0] for c in CAPACITY])
@pytest.mark.parametrize("schedule", ["auto", "fused", "two_stage", "split"])
def test_capacity_matches_compact_layout(case, schedule):
    name, B, H, Hkv, Nq, N, d, C, g, K, causal, dtype, extra = case
    sched = {"auto": 0, "two_stage": 1, "fused": 2, "split": 3}[schedule]
    if sched == 1 and dtype != "bf16":
        pytest.skip("two-stage schedule is bf16-only")
    print(f"[decode-cache] capacity {name} {schedule}", flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=11)
    q = dev(x["q"], dtype)
    compact = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    reserved = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype, Ncap=N + extra)
    a = _run_all(compact, q, dev(x["k"], dtype), dev(x["v"], dtype), sched)
    b = _run_all(reserved, q, _reserved(x["k"], N + extra, dtype), _reserved(x["v"], N + extra, dtype), sched)
    for u, w in zip(a, b):
        if u is not None:
            assert torch.equal(u, w)


def test_streaming_decode_matches_oracle():
    """Grow N one token at a time in a reserved buffer: append, select (split
    schedule), attend; every step against the oracle on the first N keys."""
    B, H, Hkv, d, C, g, K = 1, 4, 2, 128, 64, 2, 8
    N0, steps, cap = 4000, 12, 4096
    G = H // Hkv
    x = inputs.random_qkv(B, H, Hkv, steps, cap, d, "bf16", seed=5)
    kd, vd = dev(x["k"], "bf16"), dev(x["v"], "bf16")
    p = pisa.make_problem(B, H, Hkv, 1, N0, d, C, g, K, 1, "bf16", Ncap=cap)
    pyr = pisa.build_pyramid(p, kd)
    n = N0
    for s in range(steps):
        N = N0 + 1 + s
        p = pisa.make_problem(B, H, Hkv, 1, N, d, C, g, K, 1, "bf16", Ncap=cap)
        pisa.pisa_pyramid_append(p, kd, pyr, n)
        n = N
        q = dev(x["q"][:, :, s:s + 1], "bf16")
        idx = pisa.select(p, q, kd, pyr)
        o, lse = pisa.sparse_attn_fwd(p, q, kd, vd, idx)
        torch.cuda.synchronize()
        idx_np = idx.cpu().numpy()
        for h in range(Hkv):
            kh = x["k"][0, h, :N]
            levels = O.build_pyramid(kh, C, g)
            sel, gap = O.select_row(x["q"][0, h * G:(h + 1) * G, s], kh, levels, N - 1, C, g, K, True)
            if gap > 1e-3:
                assert list(idx_np[0, h, 0]) == sel + [-1] * (K - len(sel)), (s, h)
            for hq in range(h * G, (h + 1) * G):
                wo, wl = O.attention_row(x["q"][0, hq, s], kh, x["v"][0, h, :N], idx_np[0, h, 0], N - 1, C, True)
                assert np.abs(o[0, hq, 0].float().cpu().numpy() - wo).max() <= 2e-2, (s, hq)
                assert abs(float(lse[0, hq, 0]) - wl) <= 1e-3, (s, hq)
