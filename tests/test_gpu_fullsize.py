"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (automatic schedule, preallocated outputs), on sampled rows the oracle
computes one by one, plus properties that hold for every row.

Sampled rows: 512 per workload (the first and last rows, evenly spaced rows,
random rows and, for the needle workload, rows whose query was planted next to
the needle direction), checked on every KV head: indices identical to the
oracle's on decisive rows and admissible on near-tie rows (exact ties to the
smaller index), block scores against the oracle's raw-key scores, attention of
every query head of the group on the GPU's indices, and the flat baseline.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import check_flat_bsa_rows, check_selection_rows, check_valid_all_rows, pyramid_error_bound

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None

ROWS_PER_HEAD = 512


def _sample_rows(w, n=ROWS_PER_HEAD, seed=0):
    Nq = w["Nq"]
    r = np.random.default_rng(seed)
    rows = {0, 1, 2, Nq - 2, Nq - 1}
    rows |= set(np.linspace(0, Nq - 1, n // 2).astype(int).tolist())
    if w["dist"] == "needles":
        qpos = inputs.needle_layout(w)["qpos"]
        rows |= set(r.choice(qpos, size=n // 4, replace=False).tolist())
    while len(rows) < min(n, Nq):
        rows.add(int(r.integers(Nq)))
    return np.array(sorted(rows))


def _run(w, x):
    B, H, Hkv, N, Nq, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    tdt = torch.bfloat16 if w["dtype"] == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(x[n]).to(tdt).cuda() for n in "qkv")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, w["causal"], w["dtype"])
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    bsa = pisa.select_flat_bsa(p, q, pyr)
    idx2, sc = pisa.select(p, q, k, pyr, with_score=True)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2), "block_score output changed the selection"
    return pyr, idx, sc, o, lse, bsa


@pytest.mark.parametrize("name", ["gqa-32k", "needles-128k", "ar1-512k", "paper-sel-128k"])
def test_fullsize_workload(name):
    w = inputs.workload(name)
    B, H, Hkv, N, Nq, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    causal = bool(w["causal"])
    print(f"[fullsize] {name}: generating inputs", flush=True)
    x = inputs.make_inputs(w, seed=0)
    print(f"[fullsize] {name}: running the HIP path", flush=True)
    pyr, idx, sc, o, lse, bsa = _run(w, x)
    check_valid_all_rows(idx, N, Nq, C, K, causal)
    check_valid_all_rows(bsa, N, Nq, C, K, causal)
    assert torch.equal(torch.isneginf(sc), idx < 0)
    rows = _sample_rows(w)
    idx_np, sc_np, bsa_np = idx.cpu().numpy(), sc.cpu().numpy(), bsa.cpu().numpy()
    o_np, lse_np = o.float().cpu().numpy(), lse.cpu().numpy()
    sizes = O.level_sizes(N, C, g)
    offs = np.concatenate([[0], np.cumsum(sizes[:-1])])
    G = H // Hkv
    total = {}
    total_bsa = {}
    for h in range(Hkv):
        print(f"[fullsize] {name}: oracle on {len(rows)} rows of KV head {h}", flush=True)
        kh = x["k"][0, h].astype(np.float64)
        levels = O.build_pyramid(kh, C, g)
        # pyramid: every level's first, middle and last nodes
        got_pyr = pyr[0, h].cpu().numpy()
        bound = pyramid_error_bound(x["k"][:, h:h + 1], C, g, levels_of={(0, 0): levels})[0, 0]
        for lv, S in enumerate(levels[:-1] if len(levels) > 1 else levels, start=1):
            for i in sorted({0, S.shape[0] // 2, S.shape[0] - 1}):
                err = np.abs(got_pyr[offs[lv - 1] + i] - S[i])
                assert np.all(err <= bound[offs[lv - 1] + i]), (lv, i, float(err.max()))
        st = check_selection_rows(x["q"], x["k"], C, g, K, causal, idx_np[:, h:h + 1][:, :, rows], rows,
                                  gpu_score=sc_np[:, h:h + 1][:, :, rows], heads=[h], levels={(0, h): levels})
        for key, val in st.items():
            total[key] = total.get(key, 0) + val
        # attention on the GPU's indices, every head of the group
        for hq in range(h * G, (h + 1) * G):
            for r in rows:
                t = N - Nq + r
                wo, wl = O.attention_row(x["q"][0, hq, r], kh, x["v"][0, h], idx_np[0, h, r], t, C, causal)
                assert np.abs(o_np[0, hq, r] - wo).max() <= 2e-2, (h, hq, r)
                assert abs(float(lse_np[0, hq, r]) - wl) <= 1e-3, (h, hq, r)
        stb = check_flat_bsa_rows(x["q"], x["k"], C, K, causal, bsa_np[:, h:h + 1][:, :, rows], rows, heads=[h])
        for key, val in stb.items():
            total_bsa[key] = total_bsa.get(key, 0) + val
    print(f"[fullsize] {name}: selection {total}", flush=True)
    print(f"[fullsize] {name}: flat BSA {total_bsa}", flush=True)
    assert total["rows"] >= ROWS_PER_HEAD * Hkv


def test_fullsize_decode_steps():
    """Decode: 64 single-token steps against one pyramid built once; every
    step's selection, block scores and attention against the oracle."""
    w = inputs.workload("decode-128k")
    B, H, Hkv, N, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "d", "C", "g", "K"))
    x0 = inputs.make_inputs(w, seed=0, step=0)
    k = torch.from_numpy(x0["k"]).to(torch.bfloat16).cuda()
    v = torch.from_numpy(x0["v"]).to(torch.bfloat16).cuda()
    p = pisa.make_problem(B, H, Hkv, 1, N, d, C, g, K, 1, "bf16")
    pyr = pisa.build_pyramid(p, k)
    levels = {(0, h): O.build_pyramid(x0["k"][0, h].astype(np.float64), C, g) for h in range(Hkv)}
    total = {}
    for step in range(64):
        xs = inputs.make_inputs(w, seed=0, step=step, parts="q")
        q = torch.from_numpy(xs["q"]).to(torch.bfloat16).cuda()
        idx = pisa.select(p, q, k, pyr)
        o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
        idx2, sc = pisa.select(p, q, k, pyr, with_score=True)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx2)
        idx_np = idx.cpu().numpy()
        st = check_selection_rows(xs["q"], x0["k"], C, g, K, True, idx_np, [0], gpu_score=sc.cpu().numpy(),
                                  levels=levels)
        for key, val in st.items():
            total[key] = total.get(key, 0) + val
        for h in range(Hkv):
            wo, wl = O.attention_row(xs["q"][0, h, 0], x0["k"][0, h], x0["v"][0, h], idx_np[0, h, 0], N - 1, C, True)
            assert np.abs(o[0, h, 0].float().cpu().numpy() - wo).max() <= 2e-2
            assert abs(float(lse[0, h, 0]) - wl) <= 1e-3
    print(f"[fullsize] decode-128k: selection {total}", flush=True)
