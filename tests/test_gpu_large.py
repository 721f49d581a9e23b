"""Two-stage selection on a problem with more (row, leaf candidate) pairs than
a 32-bit count holds: 16 KV heads x 1,179,648 query rows x 125 scored
candidates per row is ~2.36e9 pairs.  The library runs it as passes over
(batch, KV head) slices (14 heads, then 2); the selection of heads in both
passes is checked against the oracle on sampled rows, every row for validity.
"""
import numpy as np
import pytest
import torch

from paper_2609_31093_amd import inputs
import oracle as O
from tests.helpers import check_selection_row, check_valid_all_rows

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None


def test_two_stage_beyond_2_31_pairs():
    B, H, Hkv, d, C, g, K = 1, 16, 16, 64, 128, 2, 64
    N = Nq = 9216 * C  # 9216 leaf blocks (the two-stage schedule takes up to 16384)
    assert B * Hkv * Nq * (g * K - 3) > 2 ** 31
    checked = (0, 13, 14, 15)  # the first pass holds heads 0..13, the second 14..15
    q = torch.empty((B, H, Nq, d), dtype=torch.bfloat16, device="cuda")
    k = torch.empty((B, Hkv, N, d), dtype=torch.bfloat16, device="cuda")
    rows = np.unique(np.concatenate([[0, 1, Nq // 2, Nq - 2, Nq - 1],
                                     np.random.default_rng(1).choice(Nq, 3, replace=False)]))
    host_k, host_q = {}, {}
    print("[large] generating inputs", flush=True)
    for h in range(Hkv):
        r = np.random.default_rng(np.random.SeedSequence([31, h]))
        qh = inputs.round_to_bf16(r.standard_normal((Nq, d), dtype=np.float32))
        kh = inputs.round_to_bf16(r.standard_normal((N, d), dtype=np.float32))
        q[0, h] = torch.from_numpy(qh).to(torch.bfloat16)
        k[0, h] = torch.from_numpy(kh).to(torch.bfloat16)
        if h in checked:
            host_k[h] = kh
            host_q[h] = qh[rows]
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16")
    print("[large] selection", flush=True)
    pyr = pisa.build_pyramid(p, k)
    idx, sc = pisa.select(p, q, k, pyr, with_score=True)
    torch.cuda.synchronize()
    check_valid_all_rows(idx, N, Nq, C, K, True)
    assert torch.equal(torch.isneginf(sc), idx < 0)
    print("[large] oracle", flush=True)
    idx_np = idx[0, list(checked)][:, rows].cpu().numpy()
    sc_np = sc[0, list(checked)][:, rows].cpu().numpy()
    del q, k, pyr, idx, sc
    torch.cuda.empty_cache()
    for j, h in enumerate(checked):
        kh = host_k[h].astype(np.float64)
        levels = O.build_pyramid(kh, C, g)
        other = 0
        for ri, r in enumerate(rows):
            _, o, _ = check_selection_row(host_q[h][ri:ri + 1], kh, levels, int(r), C, g, K, True, idx_np[j, ri],
                                          sc_np[j, ri], where=(h, int(r)))
            other += o
        print(f"[large] KV head {h}: {len(rows)} rows match the oracle ({other} other admissible)", flush=True)
