"""GPU parity on seeded random shapes drawn from the supported envelope (head
dim 64 / 128, leaf blocks of 32-128 keys, fan-out 2-4, 1-16 query heads per KV
head, budgets up to g*K = 128, causal or not, suffix query rows), through the
automatic schedule: indices against the oracle on sampled rows (decisive rows
identical), every row a valid selection, and attention on the GPU's own
indices within the bf16 / fp32 bounds of the other parity tests."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import check_selection_valid, compare_selection, dev

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
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    check_selection_valid(idx_np, N, Nq, C, K, bool(causal))
    rows = _rows(Nq, i)
    ora, gap = O.select(x["q"], x["k"], C, g, K, bool(causal), rows=rows)
    print(compare_selection(idx_np[:, :, rows], ora, gap))
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, bool(causal), rows=rows)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.abs(o.float().cpu().numpy()[:, :, rows] - want_o).max() <= tol
    assert np.abs(lse.cpu().numpy()[:, :, rows] - want_lse).max() <= 1e-3
