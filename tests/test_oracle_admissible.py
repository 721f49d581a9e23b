"""Pins of the oracle's near-tie admissibility check (``selection_admissible``,
``flat_bsa_admissible``): the acceptance rule for rows whose ranking margins
are within the rounding tolerance, where several selections are correct.

The check is pinned against (a) the oracle's own exact selection (always
admissible; with tol = 0 the only admissible set), (b) a second, differently
structured walk of the hierarchy that decides every ranking on scores moved by
random amounts below tol/2 (always admissible), (c) constructed exact ties
(both orders admissible without the tie rule, only the smaller index with it),
including a tie at an intermediate level whose two branches lead to different
leaf sets, and (d) planted wrong blocks (always rejected).
"""
import numpy as np
import pytest

import oracle as O

TOL = 1e-3


def _case(seed, N, d, G, scale=1.0):
    r = np.random.default_rng(seed)
    return r.standard_normal((G, d)) * scale, r.standard_normal((N, d))


def _perturbed_walk(qg, k, levels, t, C, g, K, causal, rng, amp):
    """Coarse-to-fine selection (Sec. 3.2 eq. hierarchical_topk, App. B policy)
    written as a breadth-first walk over explicit node sets, with every score
    moved by a uniform amount in [-amp, amp] before ranking."""
    M = [lv.shape[0] for lv in levels]
    f_leaf = O.forced_leaves(t, C, causal)
    kept = {0}
    for lv in range(len(M), 0, -1):
        if lv < len(M):
            span = C * g ** (lv - 1)
            kept_above = kept
            kept = set()
            cand = sorted(r for i in kept_above for r in range(i * g, min((i + 1) * g, M[lv - 1]))
                          if not causal or r * span <= t)
        else:
            cand = [0]
        forced = {j // g ** (lv - 1) for j in f_leaf} & set(cand)
        if len(cand) <= K:
            kept = set(cand)
            continue
        free = [i for i in cand if i not in forced]
        noisy = {i: O.candidate_score(qg, k, levels, lv, i, C, g) + rng.uniform(-amp, amp) for i in free}
        best = sorted(free, key=lambda i: (-noisy[i], i))[:K - len(forced)]
        kept = forced | set(best)
    return sorted(kept)


SHAPES = [(300, 4, 2, 5, 1, True), (511, 8, 4, 6, 2, True), (450, 8, 2, 8, 1, False),
          (700, 4, 3, 6, 4, True), (1024, 8, 2, 7, 2, True)]


@pytest.mark.parametrize("N,C,g,K,G,causal", SHAPES)
def test_exact_selection_is_admissible_and_unique_at_zero_tolerance(N, C, g, K, G, causal):
    qg, k = _case(N + K, N, 8, G, scale=1.5)
    levels = O.build_pyramid(k, C, g)
    for t in sorted({N // 4, N // 2, N - 1, 3 * C + 1}):
        sel, gap = O.select_row(qg, k, levels, t, C, g, K, causal)
        res = O.selection_admissible(qg, k, levels, t, C, g, K, causal, sel, tol=TOL)
        assert res["ok"] is True, (t, res)
        assert O.selection_admissible(qg, k, levels, t, C, g, K, causal, sel, tol=0.0)["ok"] is True
        # a selection short of one block is never admissible (also where no level was ranked)
        assert O.selection_admissible(qg, k, levels, t, C, g, K, causal, sel[:-1], tol=TOL)["ok"] is False
        # any one-block change of a ranked selection is rejected at tol = 0
        M1 = levels[0].shape[0]
        elig = [i for i in range(M1) if not causal or i * C <= t]
        others = [i for i in elig if i not in sel]
        forced = O.forced_leaves(t, C, causal)
        free_kept = [i for i in sel if i not in forced]
        if others and free_kept and len(elig) > K:
            wrong = sorted((set(sel) - {free_kept[0]}) | {others[0]})
            assert O.selection_admissible(qg, k, levels, t, C, g, K, causal, wrong, tol=0.0)["ok"] is False


@pytest.mark.parametrize("N,C,g,K,G,causal", SHAPES)
def test_perturbed_walk_is_always_admissible(N, C, g, K, G, causal):
    """Rankings decided on scores within tol/2 of the exact ones: the walk's
    result is accepted on every row, including rows where it differs from the
    exact selection.  Scaled-down queries make near-ties common."""
    qg, k = _case(7 * N + K, N, 8, G, scale=0.01)
    levels = O.build_pyramid(k, C, g)
    rng = np.random.default_rng(N)
    differ = 0
    for t in range(N // 3, N, max(1, N // 80)):
        exact, gap = O.select_row(qg, k, levels, t, C, g, K, causal)
        got = _perturbed_walk(qg, k, levels, t, C, g, K, causal, rng, TOL / 2)
        differ += got != exact
        res = O.selection_admissible(qg, k, levels, t, C, g, K, causal, got, tol=TOL)
        assert res["ok"] is True, (t, got, exact, gap, res["visits"])
        if gap > TOL:
            assert got == exact
    assert differ > 0, "the scale should produce near-ties that the walk resolves differently"


def test_planted_wrong_block_is_rejected_on_near_tie_rows():
    """A block far below the cut never becomes admissible, even on rows whose
    margins are within the tolerance elsewhere."""
    N, C, g, K, G = 1024, 8, 2, 7, 2
    qg, k = _case(5, N, 8, G, scale=0.05)
    levels = O.build_pyramid(k, C, g)
    checked = 0
    for t in range(N // 2, N, 16):
        trace = []
        sel, gap = O.select_row(qg, k, levels, t, C, g, K, True, trace=trace)
        leaf = trace[-1]
        if not leaf["u"] or gap > TOL:
            continue
        u = leaf["u"]
        dropped = sorted((i for i in u if i not in sel), key=lambda i: u[i])
        kept = [i for i in sel if i in u]
        worst = dropped[0]
        if u[max(kept, key=lambda i: u[i])] - u[worst] <= 10 * TOL or u[min(kept, key=lambda i: u[i])] - u[worst] <= TOL:
            continue
        wrong = sorted((set(sel) - {kept[0]}) | {worst})
        assert O.selection_admissible(qg, k, levels, t, C, g, K, True, wrong, tol=TOL)["ok"] is False
        # a block that was never a leaf candidate (its ancestors were pruned) is rejected too
        never = [i for i in range(t // C + 1) if i not in leaf["A"]]
        if never:
            wrong2 = sorted((set(sel) - {kept[0]}) | {never[0]})
            assert O.selection_admissible(qg, k, levels, t, C, g, K, True, wrong2, tol=TOL)["ok"] is False
        checked += 1
    assert checked >= 3


def test_exact_leaf_tie_both_orders_without_tie_rule():
    """Two identical key blocks competing for the last slot: both choices are
    admissible, and the tie rule R4 accepts only the smaller index."""
    N, C, g, d = 512, 8, 2, 8
    r = np.random.default_rng(3)
    q = r.standard_normal((1, d))
    k = r.standard_normal((N, d)) * 0.01
    strong = 5.0 * q[0] / np.linalg.norm(q[0])
    twins = [20, 21]          # siblings: one parent, so the tie is at the leaf level only
    for b in twins:
        k[b * C:(b + 1) * C] = strong
    levels = O.build_pyramid(k, C, g)
    t = N - 1
    c = t // C
    K = 4                     # three forced blocks + one slot for the twins
    sel, gap = O.select_row(q, k, levels, t, C, g, K, True)
    assert sel == sorted({0, c - 1, c, 20}) and gap == 0.0
    alt = sorted({0, c - 1, c, 21})
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, sel)["ok"] is True
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, alt)["ok"] is False
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, alt, strict_ties=False)["ok"] is True
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, sel, strict_ties=False)["ok"] is True


def test_intermediate_tie_branches_lead_to_different_leaves():
    """An exact tie between two level-3 nodes whose subtrees are copies, with
    one free slot at that level: the leaf below either branch is admissible
    without the tie rule (the search has to take the other branch three levels
    up to reach it), only the smaller node's with it, and a leaf that neither
    branch leads to is rejected."""
    N, C, g, d = 512, 8, 2, 8
    r = np.random.default_rng(11)
    q = r.standard_normal((1, d))
    k = r.standard_normal((N, d)) * 0.01
    span3 = C * 4                                  # tokens under one level-3 node
    a, b = 3, 9                                    # two level-3 nodes, far from the forced blocks
    pattern = r.standard_normal((span3, d)) * 0.3 + 2.0 * q[0] / np.linalg.norm(q[0])
    k[a * span3:(a + 1) * span3] = pattern
    k[b * span3:(b + 1) * span3] = pattern
    levels = O.build_pyramid(k, C, g)
    t = 60 * C + 3                                 # c = 60: forced leaves 0, 59, 60 have three level-3 ancestors
    c = t // C
    forced = {0, c - 1, c}
    K = 4                                          # one free slot at levels 3, 2 and 1
    sel, gap = O.select_row(q, k, levels, t, C, g, K, True)
    assert gap == 0.0
    free = [i for i in sel if i not in forced]
    assert len(free) == 1 and a * 4 <= free[0] < (a + 1) * 4, sel
    mirror = sorted(forced | {free[0] - a * 4 + b * 4})
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, sel)["ok"] is True
    assert O.selection_admissible(q, k, levels, t, C, g, K, True, mirror)["ok"] is False
    res = O.selection_admissible(q, k, levels, t, C, g, K, True, mirror, strict_ties=False)
    assert res["ok"] is True and res["leaf_ranked"] and res["visits"] > 4
    for other in (5, 20, 58):                      # leaves outside both branches
        wrong = sorted(forced | {other})
        assert O.selection_admissible(q, k, levels, t, C, g, K, True, wrong, strict_ties=False)["ok"] is False


def test_leaf_scores_of_the_accepted_path_are_raw_key_lse():
    """The accepted path's leaf scores are the grouped raw-key LSE (eq.
    direct_child_lse at the leaf level), the values block_score reports."""
    from scipy.special import logsumexp

    N, C, g, K, G = 600, 8, 2, 6, 2
    qg, k = _case(21, N, 8, G, scale=1.0)
    levels = O.build_pyramid(k, C, g)
    t = N - 1
    sel, _ = O.select_row(qg, k, levels, t, C, g, K, True)
    res = O.selection_admissible(qg, k, levels, t, C, g, K, True, sel)
    assert res["ok"] and res["leaf_ranked"]
    for i, u in res["leaf_u"].items():
        want = sum(logsumexp(k[i * C:(i + 1) * C] @ qh / np.sqrt(8)) for qh in qg)
        assert abs(u - want) < 1e-12


def test_flat_bsa_admissible():
    N, C, K, G = 800, 8, 6, 3
    qg, k = _case(8, N, 8, G, scale=0.02)
    S1 = O.build_pyramid(k, C, 2)[0]
    near = 0
    for t in range(N // 2, N, 25):
        sel, gap = O.flat_bsa_row(qg, S1, t, C, K, True)
        assert O.flat_bsa_admissible(qg, S1, t, C, K, True, sel)
        c = t // C
        others = [i for i in range(c + 1) if i not in sel]
        free_kept = [i for i in sel if i not in {0, c - 1, c}]
        assert not O.flat_bsa_admissible(qg, S1, t, C, K, True, sel[:-1] + [-1])
        if gap <= TOL:
            near += 1
        elif others and free_kept:
            wrong = sorted((set(sel) - {free_kept[0]}) | {others[0]})
            assert not O.flat_bsa_admissible(qg, S1, t, C, K, True, wrong, tol=0.0)
    assert near > 0


def test_row_checker_accepts_the_oracle_and_rejects_planted_errors():
    """The GPU tests' row checker (tests/helpers.py), fed the oracle's own
    selections and scores, accepts them; a changed decisive row, a wrong block
    score and a finite score on a forced block are each rejected."""
    from tests.helpers import check_selection_rows

    B, H, Hkv, N, d, C, g, K = 1, 4, 2, 640, 8, 8, 2, 6
    r = np.random.default_rng(4)
    q = r.standard_normal((B, H, N, d))
    k = r.standard_normal((B, Hkv, N, d))
    rows = np.array([5, 100, 333, 639])
    idx, gap = O.select(q, k, C, g, K, True, rows=rows)
    sc = np.full(idx.shape, -np.inf)
    for h in range(Hkv):
        lv = O.build_pyramid(k[0, h], C, g)
        for ri, row in enumerate(rows):
            trace = []
            sel, _ = O.select_row(q[0, 2 * h:2 * h + 2, row], k[0, h], lv, row, C, g, K, True, trace=trace)
            leaf = trace[-1]
            f = O.forced_leaves(row, C, True)
            for pos, j in enumerate(sel):
                sc[0, h, ri, pos] = leaf["u"][j] if (len(leaf["A"]) > K and j not in f) else np.inf
    st = check_selection_rows(q, k, C, g, K, True, idx, rows, gpu_score=sc)
    assert st["rows"] == 8 and st["scored_blocks"] > 0
    ri = int(np.argmax(np.where(np.isfinite(gap[0, 0]), gap[0, 0], -1.0)))   # a ranked decisive row of head 0
    assert gap[0, 0, ri] > 1e-3 and rows[ri] > K * C
    bad = idx.copy()
    c = rows[ri] // C
    free_pos = [pos for pos, j in enumerate(bad[0, 0, ri]) if j not in (0, c - 1, c)]
    others = [j for j in range(c + 1) if j not in bad[0, 0, ri]]
    bad[0, 0, ri, free_pos[0]] = others[0]
    bad[0, 0, ri] = np.sort(bad[0, 0, ri])
    with pytest.raises(AssertionError):
        check_selection_rows(q, k, C, g, K, True, bad, rows, gpu_score=None)
    wrong = sc.copy()
    wrong[0, 0, ri, free_pos[0]] += 2e-3
    with pytest.raises(AssertionError):
        check_selection_rows(q, k, C, g, K, True, idx, rows, gpu_score=wrong)
    wrong = sc.copy()
    fpos = list(idx[0, 0, ri]).index(0)
    wrong[0, 0, ri, fpos] = 1.0
    with pytest.raises(AssertionError):
        check_selection_rows(q, k, C, g, K, True, idx, rows, gpu_score=wrong)
