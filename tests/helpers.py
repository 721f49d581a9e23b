"""Shared helpers of the GPU parity tests: device upload, oracle comparison
(decisive rows exact, near-tie rows admissible, block scores, validity)."""
import numpy as np
import torch


def dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.to("cuda")


def check_selection_valid(idx: np.ndarray, N: int, Nq: int, C: int, K: int, causal: bool):
    """Properties every correct selection has: ascending unique in-range indices,
    the forced blocks present, and min(K, #eligible) entries."""
    B, Hkv, R, _ = idx.shape
    M1 = -(-N // C)
    for r in range(R):
        t = N - Nq + r
        c = t // C
        elig = c + 1 if causal else M1
        want_n = min(K, elig)
        for b in range(B):
            for h in range(Hkv):
                row = idx[b, h, r]
                sel = row[row >= 0]
                assert len(sel) == want_n, (b, h, r, row)
                assert np.all(row[want_n:] == -1)
                assert np.all(np.diff(sel) > 0)
                assert sel.min() >= 0 and sel.max() < (c + 1 if causal else M1)
                if causal:
                    for f in {0, c, max(c - 1, 0)}:
                        assert f in sel, (r, f, sel)


def check_valid_all_rows(idx, N, Nq, C, K, causal):
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


def _check_scores(gs, got_sel_row, forced, leaf_ranked, leaf_u, tol, where):
    """block_score of one row: -inf at padding, +inf for blocks kept without a
    score (forced, or every block when the leaf level was not ranked), else the
    block's grouped raw-key score within tol."""
    for pos, j in enumerate(got_sel_row):
        s = float(gs[pos])
        if j < 0:
            assert s == -np.inf, (where, pos, s)
        elif leaf_ranked and j not in forced:
            assert np.isfinite(s) and abs(s - leaf_u[j]) <= tol, (where, j, s, leaf_u.get(j))
        else:
            assert s == np.inf, (where, j, s)


def check_selection_row(qg, kh, levels, t, C, g, K, causal, got_row, gs_row=None, score="lse", tol=1e-3,
                        strict_ties=True, where=None):
    """Parity of one (query position t, KV head) row of pisa_select.

    qg [G, d] the group's queries, kh [N, d] the head's keys, levels the
    oracle pyramid of kh; got_row the GPU's K indices, gs_row its K block
    scores or None.  Decisive rows (oracle margin > tol at every ranked
    level) must equal the oracle; other rows must equal it or be an
    admissible selection (O.selection_admissible: some walk whose rankings
    are off by at most tol produces them; exact ties to the smaller index,
    reading R4).  Block scores: -inf at padding, +inf for blocks kept without
    a score, otherwise the oracle's grouped raw-key score within tol.
    Returns (gap, chose_other_admissible, scored blocks checked)."""
    import oracle as O

    trace = []
    want, gap = O.select_row(qg, kh, levels, t, C, g, K, causal, trace=trace, score=score)
    got_row = np.asarray(got_row, dtype=np.int64)
    got = [int(j) for j in got_row if j >= 0]
    other = False
    if got == want:
        leaf = trace[-1]
        leaf_ranked, leaf_u = len(leaf["A"]) > K, leaf["u"]
    else:
        assert gap <= tol, f"decisive row {where} differs: gpu {got} oracle {want} gap {gap}"
        res = O.selection_admissible(qg, kh, levels, t, C, g, K, causal, got, tol=tol, score=score,
                                     strict_ties=strict_ties)
        assert res["ok"] is True, (f"near-tie row {where}: gpu {got} is not an admissible selection "
                                   f"(oracle {want}, gap {gap}, search {res})")
        other = True
        leaf_ranked, leaf_u = res["leaf_ranked"], res["leaf_u"]
    n_scored = 0
    if gs_row is not None:
        f = O.forced_leaves(t, C, causal)
        _check_scores(gs_row, got_row, f, leaf_ranked, leaf_u, tol, where)
        n_scored = sum(1 for j in got if leaf_ranked and j not in f)
    return gap, other, n_scored


def check_selection_rows(q, k, C, g, K, causal, gpu_idx, rows, gpu_score=None, score="lse", tol=1e-3,
                         heads=None, levels=None, strict_ties=True):
    """check_selection_row on sampled rows of every (batch, KV head).

    q [B,H,Nq,d], k [B,Hkv,N,d] (float32 arrays of the stored values);
    gpu_idx [B,len(heads),len(rows),K] the GPU's indices of those rows (and
    gpu_score its block_score, same shape, or None); levels an optional
    {(b, h): oracle pyramid} cache.  Returns counts of decisive / near-tie /
    exact-tie rows and of near-tie rows where the GPU chose another
    admissible selection."""
    import oracle as O

    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = H // Hkv
    heads = list(range(Hkv)) if heads is None else list(heads)
    st = {"rows": 0, "decisive": 0, "near_tie": 0, "exact_tie": 0, "near_tie_other_admissible": 0,
          "scored_blocks": 0}
    for b in range(B):
        for hi, h in enumerate(heads):
            kh = np.asarray(k[b, h], dtype=np.float64)
            lv = levels[(b, h)] if levels is not None else O.build_pyramid(kh, C, g)
            for ri, r in enumerate(rows):
                t = N - Nq + int(r)
                gs = None if gpu_score is None else gpu_score[b, hi, ri]
                gap, other, n_sc = check_selection_row(q[b, h * G:(h + 1) * G, r], kh, lv, t, C, g, K, causal,
                                                       gpu_idx[b, hi, ri], gs, score, tol, strict_ties,
                                                       where=(b, h, int(r)))
                st["rows"] += 1
                st["decisive"] += gap > tol
                st["near_tie"] += gap <= tol
                st["exact_tie"] += gap == 0
                st["near_tie_other_admissible"] += other
                st["scored_blocks"] += n_sc
    return st


def check_flat_bsa_rows(q, k, C, K, causal, gpu_idx, rows, tol=1e-3, heads=None):
    """Parity of pisa_select_flat_bsa on sampled rows: identical indices on
    decisive rows, an admissible selection (O.flat_bsa_admissible) on the
    others.  Shapes as in check_selection_rows."""
    import oracle as O

    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = H // Hkv
    heads = list(range(Hkv)) if heads is None else list(heads)
    st = {"rows": 0, "decisive": 0, "near_tie": 0, "near_tie_other_admissible": 0}
    for b in range(B):
        for hi, h in enumerate(heads):
            S1 = O.build_pyramid(np.asarray(k[b, h], dtype=np.float64), C, 2)[0]
            for ri, r in enumerate(rows):
                t = N - Nq + int(r)
                qg = q[b, h * G:(h + 1) * G, r]
                want, gap = O.flat_bsa_row(qg, S1, t, C, K, causal)
                got = [int(j) for j in gpu_idx[b, hi, ri] if j >= 0]
                st["rows"] += 1
                st["decisive"] += gap > tol
                st["near_tie"] += gap <= tol
                if got != want:
                    assert gap <= tol, f"decisive flat-BSA row {(b, h, int(r))} differs: gpu {got} oracle {want}"
                    assert O.flat_bsa_admissible(qg, S1, t, C, K, causal, got, tol=tol), \
                        f"flat-BSA row {(b, h, int(r))}: gpu {got} not admissible (oracle {want}, gap {gap})"
                    st["near_tie_other_admissible"] += 1
    return st


def pyramid_error_bound(k, C, g, levels_of=None):
    """Per-element bound on |float32 pyramid - exact pyramid|, in the layout of
    oracle.pyramid ([B, Hkv, R, d]).

    Every node is a float32 mean: the sum of its n inputs in any order errs by
    at most gamma_{n-1} * sum |x| (gamma_m = m u / (1 - m u), u = 2^-24), and
    the division (or multiplication by a rounded 1/n) adds at most 2u of the
    result.  A leaf's inputs are exact (bf16 or fp32 keys); a coarser node's
    are its children as computed, each off by at most its own bound B_j, so
    the node's bound is max_j B_j (the mean of the perturbations) plus
    gamma_{n-1} * mean_j (|x_j| + B_j) plus 3u (|mean| + max_j B_j).  The
    magnitudes come from the exact (float64) pyramid of the oracle
    (levels_of: {(b, h): oracle.build_pyramid levels} already at hand)."""
    import oracle as O

    u = 2.0 ** -24
    gam = lambda n: n * u / (1.0 - n * u)
    k = np.asarray(k, dtype=np.float64)
    B, Hkv, N, d = k.shape
    out = None
    for b in range(B):
        for h in range(Hkv):
            levels = levels_of[(b, h)] if levels_of and (b, h) in levels_of else O.build_pyramid(k[b, h], C, g)
            M1 = levels[0].shape[0]
            kabs = np.zeros((M1 * C, d))
            kabs[:N] = np.abs(k[b, h])
            cnt = np.minimum(C, N - np.arange(M1) * C).astype(np.float64)
            absmean = kabs.reshape(M1, C, d).sum(axis=1) / cnt[:, None]
            bounds = [gam(cnt - 1)[:, None] * absmean + 3 * u * np.abs(levels[0])]
            for lv in range(1, len(levels)):
                cb, cx = bounds[-1], np.abs(levels[lv - 1])
                M = levels[lv].shape[0]
                nc = np.minimum(g, cb.shape[0] - np.arange(M) * g).astype(np.float64)
                pb = np.zeros((M * g, d))
                px = np.zeros((M * g, d))
                pb[:cb.shape[0]] = cb
                px[:cb.shape[0]] = cx
                bmax = pb.reshape(M, g, d).max(axis=1)
                mabs = (px + pb).reshape(M, g, d).sum(axis=1) / nc[:, None]
                bounds.append(bmax + gam(nc - 1)[:, None] * mabs + 3 * u * (np.abs(levels[lv]) + bmax))
            rows = O.pyramid_rows(bounds)
            if out is None:
                out = np.empty((B, Hkv, rows.shape[0], d))
            out[b, h] = rows
    return out
