"""GPU parity on seeded random shapes drawn from the supported envelope (head
dim 64 / 128, leaf blocks of 32-128 keys, fan-out 2-4, 1-16 query heads per KV
head, budgets up to g*K = 128, causal or not, suffix query rows), through the
automatic schedule: indices against the oracle on sampled rows (decisive rows
identical, near-tie rows admissible), block scores against the oracle's,
every row a valid selection, and attention on the GPU's own
indices within the bf16 / fp32 bounds of the other parity tests."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import check_flat_bsa_rows, check_selection_rows, check_selection_valid, dev

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None


def _shapes(n=14, seed=2024):
    r = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        d = int(r.choice([64, 128]))
        C = int(r.choice([32, 64, 96, 128]))
        g = int(r.choice([2, 3, 4]))
        G = int(r.choice([1, 2, 4, 8, 16]))
        Hkv = int(r.choice([1, 2]))
        B = int(r.choice([1, 2]))
        causal = int(r.choice([0, 1]))
        kmax = min(128 // g, 2048 // (g * g * G))
        if kmax < 3:
            continue
        K = int(r.integers(3, kmax + 1))
        N = int(r.integers(C * (K + 2), 7000))
        Nq = N if r.random() < 0.6 else int(r.integers(1, N + 1))
        dtype = "bf16" if r.random() < 0.8 else "f32"
        if B * G * Hkv * Nq * N > 2.5e9:  # keep the oracle's attention within seconds
            continue
        out.append((B, G * Hkv, Hkv, Nq, N, d, C, g, K, causal, dtype))
    return out


SHAPES = _shapes()


def _rows(Nq, seed):
    if Nq <= 64:
        return np.arange(Nq)
    r = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, 1, Nq - 1], r.choice(Nq, 40, replace=False)]))


@pytest.mark.parametrize("i", range(len(SHAPES)), ids=[f"rand{i}" for i in range(len(SHAPES))])
def test_random_shape_parity(i):
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = SHAPES[i]
    print("shape", SHAPES[i], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=100 + i)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    q, k, v = dev(x["q"], dtype), dev(x["k"], dtype), dev(x["v"], dtype)
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    idx2, sc = pisa.select(p, q, k, pyr, with_score=True)
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    assert np.array_equal(idx_np, idx2.cpu().numpy())
    check_selection_valid(idx_np, N, Nq, C, K, bool(causal))
    rows = _rows(Nq, i)
    print(check_selection_rows(x["q"], x["k"], C, g, K, bool(causal), idx_np[:, :, rows], rows,
                               gpu_score=sc.cpu().numpy()[:, :, rows]))
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, bool(causal), rows=rows)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.abs(o.float().cpu().numpy()[:, :, rows] - want_o).max() <= tol
    assert np.abs(lse.cpu().numpy()[:, :, rows] - want_lse).max() <= 1e-3


def _bf16_shapes(n, seed, nmax, kcap, nqmax=None, work=None):
    r = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        d = int(r.choice([64, 128]))
        C = int(r.choice([32, 64, 96, 128]))
        g = int(r.choice([2, 3, 4]))
        G = int(r.choice([1, 2, 4, 8]))
        Hkv = int(r.choice([1, 2]))
        causal = int(r.choice([0, 1]))
        kmax = min(kcap, 128 // g, 2048 // (g * g * G), nmax // C - 2)
        if kmax < 3:
            continue
        K = int(r.integers(3, kmax + 1))
        N = int(r.integers(C * (K + 2), nmax + 1))
        Nq = N if r.random() < 0.6 else int(r.integers(1, N + 1))
        if nqmax:
            Nq = min(Nq, nqmax)
        if work and G * Hkv * Nq * K * C * d > work:  # keep the oracle within seconds
            continue
        out.append((1, G * Hkv, Hkv, Nq, N, d, C, g, K, causal, "bf16"))
    return out


SCHED_SHAPES = _bf16_shapes(8, 7, 5000, 40)


@pytest.mark.parametrize("schedule", (2, 1, 3), ids=["fused", "two_stage", "split"])
@pytest.mark.parametrize("i", range(len(SCHED_SHAPES)), ids=[f"rs{i}" for i in range(len(SCHED_SHAPES))])
def test_random_shape_schedules(i, schedule):
    """Every schedule, forced, on further random bf16 shapes."""
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = SCHED_SHAPES[i]
    print("shape", SCHED_SHAPES[i], "schedule", schedule, flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=200 + i)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype, schedule)
    q, k = dev(x["q"], dtype), dev(x["k"], dtype)
    idx, sc = pisa.select(p, q, k, pisa.build_pyramid(p, k), with_score=True)
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    check_selection_valid(idx_np, N, Nq, C, K, bool(causal))
    rows = _rows(Nq, 50 + i)
    print(check_selection_rows(x["q"], x["k"], C, g, K, bool(causal), idx_np[:, :, rows], rows,
                               gpu_score=sc.cpu().numpy()[:, :, rows]))


BWD_SHAPES = _bf16_shapes(6, 11, 2400, 48, nqmax=1200, work=6e8)


@pytest.mark.parametrize("i", range(len(BWD_SHAPES)), ids=[f"rb{i}" for i in range(len(BWD_SHAPES))])
def test_random_shape_backward(i):
    """Backward with the GPU's own selection against the float64 oracle: every
    gradient within 2% of its tensor's scale (the bound of the backward
    parity tests)."""
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = BWD_SHAPES[i]
    print("shape", BWD_SHAPES[i], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=300 + i)
    do_np = inputs.round_to_bf16(np.random.default_rng(400 + i).standard_normal((B, H, Nq, d)).astype(np.float32))
    q, k, v = (dev(x[n], dtype) for n in "qkv")
    d_o = dev(do_np, dtype)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    torch.cuda.synchronize()
    want = O.sparse_attention_bwd(x["q"], x["k"], x["v"], idx.cpu().numpy(), do_np, C, bool(causal))
    for label, got, w in zip(("dq", "dk", "dv"), (dq, dk, dv), want):
        scale = float(np.abs(w).max())
        err = float(np.abs(got.float().cpu().numpy() - w).max())
        assert err <= 2e-2 * scale, (label, err, scale)


QUAL_SHAPES = _bf16_shapes(6, 13, 4000, 64)


@pytest.mark.parametrize("i", range(len(QUAL_SHAPES)), ids=[f"rq{i}" for i in range(len(QUAL_SHAPES))])
def test_random_shape_quality(i):
    """Selection-quality diagnostic against the oracle on sampled rows: the
    reference set identical where it is decided by more than 1e-5 of mass,
    Recall@K exact there, mass figures within 1e-4."""
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = QUAL_SHAPES[i]
    print("shape", QUAL_SHAPES[i], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=500 + i)
    q, k = dev(x["q"], dtype), dev(x["k"], dtype)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    rows = _rows(Nq, 60 + i)
    met, ref = pisa.selection_quality(p, q, k, idx, torch.from_numpy(rows.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    want_met, want_ref, gap = O.selection_quality(x["q"], x["k"], idx.cpu().numpy()[:, :, rows], C, K,
                                                  bool(causal), rows)
    got_met, got_ref = met.cpu().numpy(), ref.cpu().numpy()
    decisive = gap > 1e-5
    assert not ((got_ref != want_ref).any(-1) & decisive).any()
    np.testing.assert_array_equal(np.rint(got_met[..., 0] * K)[decisive], np.rint(want_met[..., 0] * K)[decisive])
    np.testing.assert_allclose(got_met[..., 1:], want_met[..., 1:], atol=1e-4, rtol=0)


BSA_SHAPES = [s for s in _shapes(10, 31) if s[8] <= 32]


@pytest.mark.parametrize("i", range(len(BSA_SHAPES)), ids=[f"rf{i}" for i in range(len(BSA_SHAPES))])
def test_random_shape_flat_bsa(i):
    """Flat block selection (the baseline) against its oracle on sampled rows."""
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = BSA_SHAPES[i]
    print("shape", BSA_SHAPES[i], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=600 + i)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    q, k = dev(x["q"], dtype), dev(x["k"], dtype)
    idx = pisa.select_flat_bsa(p, q, pisa.build_pyramid(p, k))
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    check_selection_valid(idx_np, N, Nq, C, K, bool(causal))
    rows = _rows(Nq, 70 + i)
    print(check_flat_bsa_rows(x["q"], x["k"], C, K, bool(causal), idx_np[:, :, rows], rows))


def _edge_shapes(n=16, seed=77):
    """Small and degenerate shapes: a handful of blocks (N from below one
    block to a few), single query rows, budgets at or above the block count."""
    r = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        d = int(r.choice([64, 128]))
        C = int(r.choice([32, 64, 128]))
        g = int(r.choice([2, 3, 4]))
        G = int(r.choice([1, 2, 4, 8, 16]))
        Hkv = int(r.choice([1, 2]))
        causal = int(r.choice([0, 1]))
        N = int(r.integers(1, 6 * C + 1))
        M1 = -(-N // C)
        kmax = min(128 // g, 2048 // (g * g * G), M1 + 2)
        K = int(r.integers(3, max(4, kmax + 1)))
        if g * K > 128 or g * g * K * G > 2048:
            continue
        Nq = int(r.choice([1, 2, N])) if N > 2 else N
        Nq = min(Nq, N)
        dtype = "bf16" if r.random() < 0.75 else "f32"
        out.append((1, G * Hkv, Hkv, Nq, N, d, C, g, K, causal, dtype))
    return out


EDGE_SHAPES = _edge_shapes()


@pytest.mark.parametrize("i", range(len(EDGE_SHAPES)), ids=[f"re{i}" for i in range(len(EDGE_SHAPES))])
def test_edge_shape_parity(i):
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = EDGE_SHAPES[i]
    print("shape", EDGE_SHAPES[i], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=700 + i)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    q, k, v = dev(x["q"], dtype), dev(x["k"], dtype), dev(x["v"], dtype)
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    bsa = pisa.select_flat_bsa(p, q, pyr) if K <= 32 or dtype == "f32" or N // C < 16384 else None
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    check_selection_valid(idx_np, N, Nq, C, K, bool(causal))
    rows = np.arange(Nq)
    check_selection_rows(x["q"], x["k"], C, g, K, bool(causal), idx_np, rows)
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np, C, bool(causal), rows=rows)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.abs(o.float().cpu().numpy() - want_o).max() <= tol
    assert np.abs(lse.cpu().numpy() - want_lse).max() <= 1e-3
    if bsa is not None:
        check_flat_bsa_rows(x["q"], x["k"], C, K, bool(causal), bsa.cpu().numpy(), rows)
