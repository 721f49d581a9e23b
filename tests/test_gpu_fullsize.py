"""Parity at the workloads' full sizes, in the launch configuration bench.py
times (automatic schedule, preallocated outputs), on sampled rows the oracle
computes one by one, plus properties that hold for every row.

Sampled rows per KV head: the first and last rows, evenly spaced rows, and
(needle workload) rows whose query was planted next to the needle direction.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import compare_selection

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None


def _valid_all_rows(idx, N, Nq, C, K, causal):
    """Vectorised validity of every row: ascending, unique, in range, forced
    blocks present, min(K, eligible) entries, -1 padding."""
    idx = torch.as_tensor(idx)
    t = torch.arange(N - Nq, N, device=idx.device).view(1, 1, Nq)
    c = t // C
    M1 = -(-N // C)
    elig = (c + 1) if causal else torch.full_like(c, M1)
    want_n = torch.clamp(elig, max=K)
    n = (idx >= 0).sum(-1)
    assert torch.equal(n, want_n.expand_as(n))
    pos = torch.arange(K, device=idx.device).view(1, 1, 1, K)
    assert torch.all((pos < n.unsqueeze(-1)) == (idx >= 0))
    big = torch.where(idx >= 0, idx, torch.full_like(idx, 1 << 30))
    assert torch.all((big[..., 1:] > big[..., :-1]) | (idx[..., 1:] < 0))
    hi = (c if causal else torch.full_like(c, M1 - 1)).unsqueeze(-1)
    assert torch.all((idx < 0) | (idx <= hi))
    if causal:
        for f in (torch.zeros_like(c), c, torch.clamp(c - 1, min=0)):
            assert torch.all((idx == f.unsqueeze(-1)).any(-1))


def _sample_rows(w, n_even=12, seed=0):
    Nq = w["Nq"]
    rows = {0, 1, Nq - 2, Nq - 1}
    rows |= set(np.linspace(0, Nq - 1, n_even).astype(int).tolist())
    if w["dist"] == "needles":
        qpos = inputs.needle_layout(w)["qpos"]
        r = np.random.default_rng(seed)
        rows |= set(r.choice(qpos, size=6, replace=False).tolist())
    return sorted(r for r in rows if 0 <= r < Nq)


def _run(w, x):
    B, H, Hkv, N, Nq, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    tdt = torch.bfloat16 if w["dtype"] == "bf16" else torch.float32
    q, k, v = (torch.from_numpy(x[n]).to(tdt).cuda() for n in "qkv")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, w["causal"], w["dtype"])
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    bsa = pisa.select_flat_bsa(p, q, pyr)
    torch.cuda.synchronize()
    return pyr, idx, o, lse, bsa


@pytest.mark.parametrize("name", ["gqa-32k", "needles-128k", "ar1-512k", "paper-sel-128k"])
def test_fullsize_workload(name):
    w = inputs.workload(name)
    B, H, Hkv, N, Nq, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    causal = bool(w["causal"])
    print(f"[fullsize] {name}: generating inputs", flush=True)
    x = inputs.make_inputs(w, seed=0)
    print(f"[fullsize] {name}: running the HIP path", flush=True)
    pyr, idx, o, lse, bsa = _run(w, x)
    _valid_all_rows(idx, N, Nq, C, K, causal)
    if bsa is not None:
        _valid_all_rows(bsa, N, Nq, C, K, causal)
    rows = _sample_rows(w)
    idx_np = idx.cpu().numpy()
    heads = list(range(Hkv)) if Hkv <= 4 else [0, Hkv // 2, Hkv - 1]
    sizes = O.level_sizes(N, C, g)
    offs = np.concatenate([[0], np.cumsum(sizes[:-1])])
    G = H // Hkv
    print(f"[fullsize] {name}: oracle on {len(rows)} rows x {len(heads)} KV heads", flush=True)
    stats = []
    for h in heads:
        kh = x["k"][0, h].astype(np.float64)
        levels = O.build_pyramid(kh, C, g)
        # pyramid: every level's first, middle and last nodes
        got_pyr = pyr[0, h].cpu().numpy()
        for lv, S in enumerate(levels[:-1] if len(levels) > 1 else levels, start=1):
            for i in sorted({0, S.shape[0] // 2, S.shape[0] - 1}):
                err = np.abs(got_pyr[offs[lv - 1] + i] - S[i]).max()
                assert err <= (C + len(sizes) * g) * 2.0 ** -24 * float(np.abs(kh).max()), (lv, i, err)
        want = np.full((len(rows), K), -1)
        gaps = np.zeros(len(rows))
        for ri, r in enumerate(rows):
            t = N - Nq + r
            sel, gp = O.select_row(x["q"][0, h * G:(h + 1) * G, r], kh, levels, t, C, g, K, causal)
            want[ri, :len(sel)] = sel
            gaps[ri] = gp
        stats.append(compare_selection(idx_np[0:1, h:h + 1, rows], want[None, None], gaps[None, None]))
        # attention on the GPU's indices, every head of the group
        for hq in range(h * G, (h + 1) * G):
            for ri, r in enumerate(rows):
                t = N - Nq + r
                wo, wl = O.attention_row(x["q"][0, hq, r], kh, x["v"][0, h], idx_np[0, h, r], t, C, causal)
                go = o[0, hq, r].float().cpu().numpy()
                assert np.abs(go - wo).max() <= 2e-2, (h, hq, r)
                assert abs(float(lse[0, hq, r]) - wl) <= 1e-3, (h, hq, r)
        if bsa is not None:
            S1 = levels[0]
            bsa_np = bsa[0, h].cpu().numpy()
            for r in rows:
                t = N - Nq + r
                sel, gp = O.flat_bsa_row(x["q"][0, h * G:(h + 1) * G, r], S1, t, C, K, causal)
                if gp > 1e-3:
                    assert list(bsa_np[r][bsa_np[r] >= 0]) == sel, (h, r)
    print(f"[fullsize] {name}: {stats}", flush=True)


def test_fullsize_decode_steps():
    """Decode: 64 single-token steps against one pyramid built once."""
    w = inputs.workload("decode-128k")
    B, H, Hkv, N, d, C, g, K = (w[k] for k in ("B", "H", "Hkv", "N", "d", "C", "g", "K"))
    x0 = inputs.make_inputs(w, seed=0, step=0)
    k = torch.from_numpy(x0["k"]).to(torch.bfloat16).cuda()
    v = torch.from_numpy(x0["v"]).to(torch.bfloat16).cuda()
    p = pisa.make_problem(B, H, Hkv, 1, N, d, C, g, K, 1, "bf16")
    pyr = pisa.build_pyramid(p, k)
    levels = [O.build_pyramid(x0["k"][0, h].astype(np.float64), C, g) for h in range(Hkv)]
    for step in range(0, 64, 8):
        xs = inputs.make_inputs(w, seed=0, step=step, parts="q")
        q = torch.from_numpy(xs["q"]).to(torch.bfloat16).cuda()
        idx = pisa.select(p, q, k, pyr)
        o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
        torch.cuda.synchronize()
        idx_np = idx.cpu().numpy()
        for h in range(Hkv):
            sel, gp = O.select_row(xs["q"][0, h:h + 1, 0], x0["k"][0, h], levels[h], N - 1, C, g, K, True)
            if gp > 1e-3:
                assert list(idx_np[0, h, 0]) == sel + [-1] * (K - len(sel)), (step, h)
            wo, wl = O.attention_row(xs["q"][0, h, 0], x0["k"][0, h], x0["v"][0, h], idx_np[0, h, 0], N - 1, C, True)
            assert np.abs(o[0, h, 0].float().cpu().numpy() - wo).max() <= 2e-2
            assert abs(float(lse[0, h, 0]) - wl) <= 1e-3
