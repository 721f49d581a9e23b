"""GPU parity of the block-selection quality diagnostic (pisa_selection_quality)
against the oracle's full-attention reference (Sec. 4 eq. oracle_metrics;
App. C eq. oracle_block_mass), through the C ABI.

The diagnostic is fed the GPU's own selection (pisa_select); the oracle gets
the same selection for the same rows.  The reference set must be identical on
rows whose reference is decided by more than 1e-5 of grouped mass (smaller
gaps are fp32 rounding of sums of exponentials); Recall@K is then exact, and
captured mass and mass ratio agree to 1e-4.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None

GAP_TOL = 1e-5

SHAPES = {
    # name: (B, H, Hkv, Nq, N, d, C, K, causal)
    "gqa2-c64": (1, 4, 2, 3000, 3000, 128, 64, 8, 1),
    "mha-c32-d64": (2, 2, 2, 1500, 1500, 64, 32, 6, 1),
    "gqa4-c128": (1, 8, 2, 2600, 2600, 128, 128, 5, 1),
    "noncausal-c64": (1, 2, 1, 900, 1000, 128, 64, 4, 0),
    "suffix-c96": (1, 3, 1, 400, 4000, 64, 96, 7, 1),
}


def _rows(Nq, n=40, seed=0):
    r = np.random.default_rng(seed)
    rows = set(r.choice(Nq, size=min(n, Nq), replace=False).tolist()) | {0, Nq - 1}
    return np.array(sorted(rows), dtype=np.int64)


def _check(x, p, idx, rows, met, ref, K, C, causal):
    sel = idx.cpu().numpy()[:, :, rows]
    want_met, want_ref, gap = O.selection_quality(x["q"], x["k"], sel, C, K, bool(causal), rows)
    got_met = met.cpu().numpy()
    got_ref = ref.cpu().numpy()
    decisive = gap > GAP_TOL
    bad = np.argwhere((got_ref != want_ref).any(-1) & decisive)
    assert bad.size == 0, (bad[:5], got_ref[tuple(bad[0])], want_ref[tuple(bad[0])], gap[tuple(bad[0])])
    # Recall@K = hits / K: compare the hit counts (the GPU divides in fp32)
    np.testing.assert_array_equal(np.rint(got_met[..., 0] * K)[decisive], np.rint(want_met[..., 0] * K)[decisive])
    np.testing.assert_allclose(got_met[..., 1:], want_met[..., 1:], atol=1e-4, rtol=0)
    return int(decisive.sum()), int((~decisive).sum())


@pytest.mark.parametrize("name", list(SHAPES))
def test_quality_parity(name):
    B, H, Hkv, Nq, N, d, C, K, causal = SHAPES[name]
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=3)
    q, k = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qk")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, causal, "bf16")
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    rows = _rows(Nq)
    met, ref = pisa.selection_quality(p, q, k, idx, torch.from_numpy(rows.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    n_dec, n_tie = _check(x, p, idx, rows, met, ref, K, C, causal)
    assert n_dec > 0
    print(f"{name}: decisive rows {n_dec}, near ties {n_tie}")


def test_quality_of_the_reference_is_perfect_and_bad_rows_are_flagged():
    """Feeding the diagnostic its own reference set gives Recall@K = 1 and
    mass ratio 1 on rows with more than K eligible blocks; rows outside
    [0, Nq) get NaN metrics and an empty reference."""
    B, H, Hkv, Nq, N, d, C, K = 1, 2, 1, 2000, 2000, 128, 64, 6
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=4)
    q, k = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qk")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, 1, "bf16")
    rows = np.arange(0, Nq, 37, dtype=np.int64)
    rows_d = torch.from_numpy(rows.astype(np.int32)).cuda()
    idx = torch.full((B, Hkv, Nq, K), -1, dtype=torch.int32, device="cuda")
    _, ref = pisa.selection_quality(p, q, k, idx, rows_d)
    idx[:, :, rows_d.long()] = ref
    met, ref2 = pisa.selection_quality(p, q, k, idx, rows_d)
    torch.cuda.synchronize()
    assert torch.equal(ref, ref2)
    m = met.cpu().numpy()
    many = (N - Nq + rows) // C + 1 > K
    np.testing.assert_array_equal(m[0, 0, many, 0], 1.0)
    np.testing.assert_allclose(m[0, 0, many, 2], 1.0, atol=1e-6)
    bad = torch.tensor([-1, Nq, 5], dtype=torch.int32, device="cuda")
    met_b, ref_b = pisa.selection_quality(p, q, k, idx, bad)
    torch.cuda.synchronize()
    assert torch.isnan(met_b[0, 0, :2]).all() and (ref_b[0, 0, :2] == -1).all()
    assert not torch.isnan(met_b[0, 0, 2]).any()


def test_quality_needles_128k_sample():
    """The diagnostic at the needle workload's full size, in the launch
    configuration bench.py --quality uses, on rows the oracle computes one by
    one (needle-query rows included)."""
    w = inputs.workload("needles-128k")
    x = inputs.make_inputs(w, seed=0)
    B, H, Hkv, N, Nq, d, C, g, K = (w[kk] for kk in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    q, k = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qk")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16")
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    qpos = inputs.needle_layout(w)["qpos"]
    r = np.random.default_rng(0)
    rows = np.array(sorted(set(r.choice(qpos, 3, replace=False).tolist()) | {Nq - 1, Nq // 3, 2 * Nq // 3}))
    met, ref = pisa.selection_quality(p, q, k, idx, torch.from_numpy(rows.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    sel = idx.cpu().numpy()[:, :2, rows]
    want_met, want_ref, gap = O.selection_quality(x["q"], x["k"], sel, C, K, True, rows, heads=[0, 1])
    got_met, got_ref = met.cpu().numpy()[:, :2], ref.cpu().numpy()[:, :2]
    decisive = gap > GAP_TOL
    assert not ((got_ref != want_ref).any(-1) & decisive).any()
    np.testing.assert_allclose(got_met[..., 1:], want_met[..., 1:], atol=1e-4, rtol=0)
