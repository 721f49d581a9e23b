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
* Capacity growth (pisa_cache_capacity, pisa_cache_grow): a decode stream
  that outgrows its buffers three times, and chunked appends past the
  capacity, keep the pyramid equal to a full build bit for bit and every
  step's selection and attention equal to the oracle's.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import check_selection_row, dev

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
            check_selection_row(x["q"][0, h * G:(h + 1) * G, s], kh, levels, N - 1, C, g, K, True, idx_np[0, h, 0],
                                where=(s, h))
            for hq in range(h * G, (h + 1) * G):
                wo, wl = O.attention_row(x["q"][0, hq, s], kh, x["v"][0, h, :N], idx_np[0, h, 0], N - 1, C, True)
                assert np.abs(o[0, hq, 0].float().cpu().numpy() - wo).max() <= 2e-2, (s, hq)
                assert abs(float(lse[0, hq, 0]) - wl) <= 1e-3, (s, hq)


def _stored_equal(pa, pyr_a, pb, pyr_b):
    """The stored levels of problems pa, pb (same N, any capacities) hold equal rows."""
    for (fa, n), (fb, nb) in zip(_valid_rows(pa), _valid_rows(pb)):
        assert n == nb
        if not torch.equal(pyr_a[:, :, fa:fa + n], pyr_b[:, :, fb:fb + n]):
            return False
    return True


def test_streaming_decode_across_growth():
    """A decode stream from 500 to 1200 tokens in a cache that starts with
    room for 512: the capacity rule gives 768, 1152 and 1728 at tokens 513,
    769 and 1153, and pisa_cache_grow moves the pyramid, k and v each time.
    Every step appends one token, selects and attends, all against the oracle
    on the first N keys; after each growth the moved pyramid equals the old one
    row for row and a full build at the new capacity bit for bit, and at the
    end the pyramid equals a full build at N = 1200."""
    B, H, Hkv, d, C, g, K = 1, 4, 2, 64, 32, 2, 6
    N0, N1, cap = 500, 1200, 512
    G = H // Hkv
    x = inputs.random_qkv(B, H, Hkv, N1 - N0, N1, d, "bf16", seed=23)
    kfull, vfull = dev(x["k"], "bf16"), dev(x["v"], "bf16")
    kd = torch.zeros((B, Hkv, cap, d), dtype=torch.bfloat16, device="cuda")
    vd = torch.zeros_like(kd)
    kd[:, :, :N0] = kfull[:, :, :N0]
    vd[:, :, :N0] = vfull[:, :, :N0]
    pyr = pisa.build_pyramid(pisa.make_problem(B, H, Hkv, 1, N0, d, C, g, K, 1, "bf16", Ncap=cap), kd)
    caps = [cap]
    n = N0
    for s in range(N1 - N0):
        N = n + 1
        if N > cap:
            new_cap = pisa.pisa_cache_capacity(cap, N, C)
            p_cur = pisa.make_problem(B, H, Hkv, 1, n, d, C, g, K, 1, "bf16", Ncap=cap)
            p_new, pyr_new, kd_new, vd_new = pisa.grow_cache(p_cur, new_cap, pyr, kd, vd)
            full = pisa.build_pyramid(p_new, kd_new)
            torch.cuda.synchronize()
            assert _stored_equal(p_cur, pyr, p_new, pyr_new), (n, new_cap)
            assert _stored_equal(p_new, full, p_new, pyr_new), (n, new_cap)
            assert torch.equal(kd_new[:, :, :n], kd[:, :, :n]) and torch.equal(vd_new[:, :, :n], vd[:, :, :n])
            pyr, kd, vd, cap = pyr_new, kd_new, vd_new, new_cap
            caps.append(cap)
            print(f"[decode-cache] grew to {cap} at token {N}", flush=True)
        kd[:, :, n] = kfull[:, :, n]
        vd[:, :, n] = vfull[:, :, n]
        p = pisa.make_problem(B, H, Hkv, 1, N, d, C, g, K, 1, "bf16", Ncap=cap)
        pisa.pisa_pyramid_append(p, kd, pyr, n)
        q = dev(x["q"][:, :, s:s + 1], "bf16")
        idx, sc = pisa.select(p, q, kd, pyr, with_score=True)
        o, lse = pisa.sparse_attn_fwd(p, q, kd, vd, idx)
        torch.cuda.synchronize()
        idx_np, sc_np = idx.cpu().numpy(), sc.cpu().numpy()
        o_np, lse_np = o.float().cpu().numpy(), lse.cpu().numpy()
        for h in range(Hkv):
            kh = x["k"][0, h, :N]
            levels = O.build_pyramid(kh, C, g)
            check_selection_row(x["q"][0, h * G:(h + 1) * G, s], kh, levels, N - 1, C, g, K, True, idx_np[0, h, 0],
                                sc_np[0, h, 0], where=(s, h))
            for hq in range(h * G, (h + 1) * G):
                wo, wl = O.attention_row(x["q"][0, hq, s], kh, x["v"][0, h, :N], idx_np[0, h, 0], N - 1, C, True)
                assert np.abs(o_np[0, hq, 0] - wo).max() <= 2e-2, (s, hq)
                assert abs(float(lse_np[0, hq, 0]) - wl) <= 1e-3, (s, hq)
        n = N
    assert caps == [512, 768, 1152, 1728]
    p = pisa.make_problem(B, H, Hkv, 1, N1, d, C, g, K, 1, "bf16", Ncap=cap)
    full = pisa.build_pyramid(p, kd)
    torch.cuda.synchronize()
    assert _stored_equal(p, full, p, pyr)


GROW_CHUNK = [
    # (dtype, Hkv, d, C, g, N0, cap0, N1)
    ("f32", 2, 64, 64, 3, 1000, 1024, 3000),
    ("bf16", 1, 128, 128, 4, 5000, 5120, 40000),
    ("bf16", 2, 128, 64, 2, 64, 64, 65),
]


@pytest.mark.parametrize("case", GROW_CHUNK, ids=[f"{c[0]}-C{c[3]}-g{c[4]}-{c[5]}to{c[7]}" for c in GROW_CHUNK])
def test_chunk_append_across_growth(case):
    """A chunk of tokens past the capacity: grow the pyramid alone (keys and
    values moved by the caller), append the chunk; equal to a full build bit
    for bit and to the oracle's pyramid within the pyramid tolerance."""
    dtype, Hkv, d, C, g, N0, cap0, N1 = case
    r = np.random.default_rng(N0 + N1)
    k = r.standard_normal((1, Hkv, N1, d), dtype=np.float32)
    if dtype == "bf16":
        k = inputs.round_to_bf16(k)
    p0 = pisa.make_problem(1, Hkv, Hkv, 1, N0, d, C, g, 4, 1, dtype, Ncap=cap0)
    k0 = _reserved(k[:, :, :N0], cap0, dtype)
    pyr0 = pisa.build_pyramid(p0, k0)
    new_cap = pisa.pisa_cache_capacity(cap0, N1, C)
    assert new_cap >= N1 and new_cap % C == 0
    p_mid, pyr1, kn, vn = pisa.grow_cache(p0, new_cap, pyr0)
    assert kn is None and vn is None
    k1 = _reserved(k, new_cap, dtype)       # the caller's own copy of the keys
    p1 = pisa.make_problem(1, Hkv, Hkv, 1, N1, d, C, g, 4, 1, dtype, Ncap=new_cap)
    pisa.pisa_pyramid_append(p1, k1, pyr1, N0)
    full = pisa.build_pyramid(p1, k1)
    torch.cuda.synchronize()
    assert _stored_equal(p1, full, p1, pyr1)
    want = O.pyramid(k, C, g)
    L = len(O.level_sizes(N1, C, g))
    tol = (C + L * g) * 2.0 ** -24 * float(np.abs(k).max())
    row = 0
    for first, n in _valid_rows(p1):
        assert np.abs(pyr1[:, :, first:first + n].cpu().numpy() - want[:, :, row:row + n]).max() <= tol
        row += n
