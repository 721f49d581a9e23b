"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these re-types the oracle: each compares it with a closed form, a
hand-worked fixture, an invariant the paper proves, a special case that
reduces to a library routine (scipy / torch), or a differently structured
brute force on tiny inputs.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp, softmax

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------- hierarchy ---

def test_level_sizes_golden():
    """Sec. 3.2 eq. (key_hierarchy): sizes worked out by hand."""
    with open(os.path.join(GOLDEN, "level_sizes.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        assert O.level_sizes(c["N"], c["C"], c["g"]) == c["sizes"], c


def test_pyramid_ragged_golden():
    """Sec. 3.2 eq. (mean_pyramid): mean over valid children, hand-worked."""
    with open(os.path.join(GOLDEN, "pyramid_ragged.json")) as f:
        gold = json.load(f)
    levels = O.build_pyramid(np.array(gold["keys"], float), gold["C"], gold["g"])
    assert [lv.shape[0] for lv in levels] == gold["level_sizes"]
    for got, want in zip(levels, gold["levels"]):
        np.testing.assert_array_equal(got, np.array(want, float))


@pytest.mark.parametrize("N,C,g", [(1000, 8, 2), (777, 4, 3), (4096, 64, 2), (513, 16, 4)])
def test_pyramid_complete_nodes_are_raw_means(N, C, g):
    """Sec. 3.2: with equal-size children the summary is the mean of all raw keys it covers."""
    k = _rng(1).standard_normal((N, 5))
    levels = O.build_pyramid(k, C, g)
    for lv, S in enumerate(levels, start=1):
        span = C * g ** (lv - 1)
        for i in range(S.shape[0]):
            if (i + 1) * span <= N:      # complete node: every descendant is full
                np.testing.assert_allclose(S[i], k[i * span:(i + 1) * span].mean(0),
                                           rtol=0, atol=1e-13)


def test_pyramid_rows_layout():
    k = _rng(2).standard_normal((1, 1, 300, 3))
    P = O.pyramid(k, 8, 2)
    sizes = O.level_sizes(300, 8, 2)           # 38,19,10,5,3,2,1
    assert P.shape == (1, 1, sum(sizes[:-1]), 3)
    single = O.pyramid(k[:, :, :5], 8, 2)      # one leaf block: level 1 only
    assert single.shape == (1, 1, 1, 3)


# ----------------------------------------------------------------- scoring ---

def test_lse_matches_scipy():
    z = _rng(3).standard_normal(50) * 30
    assert O.lse(z) == pytest.approx(logsumexp(z), rel=1e-14)
    assert O.lse(np.array([])) == -math.inf


def _tiny_case(seed, N, d, G, scale=1.0):
    r = _rng(seed)
    return r.standard_normal((G, d)) * scale, r.standard_normal((N, d))


def test_leaf_score_is_raw_key_logsumexp():
    """Sec. 3.2 eq. (direct_child_lse) at l = 1: exact LSE over the block's raw keys,
    summed over the grouped heads (Sec. 3.3 eq. kernel_grouped_score)."""
    N, C, g, K, d, G = 2048, 16, 2, 6, 8, 3
    qg, k = _tiny_case(4, N, d, G)
    levels = O.build_pyramid(k, C, g)
    t = N - 1
    trace = []
    O.select_row(qg, k, levels, t, C, g, K, True, trace)
    leaf = trace[-1]
    assert leaf["level"] == 1 and leaf["u"], "leaf level must be ranked here"
    for i, u in leaf["u"].items():
        want = sum(logsumexp(k[i * C:(i + 1) * C] @ qh / math.sqrt(d)) for qh in qg)
        assert u == pytest.approx(want, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_jensen_chain_on_intermediate_scores(seed):
    """App. A eq. (equal_child_jensen): for a fully visible node with g equal children,
    mean_j m_j <= s - log g <= LSE_raw(B) - log|B|, with m_j the child-mean logits."""
    N, C, g, K, d = 4096, 8, 2, 5, 6
    qg, k = _tiny_case(10 + seed, N, d, 1, scale=2.0)
    levels = O.build_pyramid(k, C, g)
    q = qg[0]
    checked = 0
    for t in (N - 1, N // 2 + 3, 1500):
        trace = []
        O.select_row(qg, k, levels, t, C, g, K, True, trace)
        for rec in trace:
            lv = rec["level"]
            if lv < 2:
                continue
            span = C * g ** (lv - 1)
            cspan = span // g
            for i, s in rec["u"].items():
                lo, hi = i * span, (i + 1) * span
                assert hi <= t + 1, "scored nodes must lie in the past"
                z = k[lo:hi] @ q / math.sqrt(d)
                m = [z[j * cspan:(j + 1) * cspan].mean() for j in range(g)]
                left = float(np.mean(m))
                mid = s - math.log(g)
                right = logsumexp(z) - math.log(hi - lo)
                assert left <= mid + 1e-12 and mid <= right + 1e-12
                checked += 1
    assert checked > 20


def test_jensen_equality_when_child_logits_equal():
    """App. A: F_hat(B) = F_q(B) when all logits within each child are equal.
    Keys constant inside every leaf block make this hold for level-2 nodes."""
    N, C, g, K, d = 2048, 8, 2, 4, 6
    r = _rng(20)
    leaf_keys = r.standard_normal((N // C, d))
    k = np.repeat(leaf_keys, C, axis=0)
    q = r.standard_normal((1, d))
    levels = O.build_pyramid(k, C, g)
    trace = []
    O.select_row(q, k, levels, N - 1, C, g, K, True, trace)
    rec = [x for x in trace if x["level"] == 2][0]
    assert rec["u"]
    for i, s in rec["u"].items():
        z = k[i * C * g:(i + 1) * C * g] @ q[0] / math.sqrt(d)
        assert s - math.log(g) == pytest.approx(logsumexp(z) - math.log(C * g), abs=1e-12)


# --------------------------------------------------------------- selection ---

@pytest.mark.parametrize("g,K", [(2, 4), (3, 5), (4, 3), (2, 8)])
def test_candidate_bound(g, K):
    """Sec. 3.2 eq. (candidate_bound): |I| <= K and |A| <= gK below the root."""
    N, C, d = 3000, 4, 8
    qg, k = _tiny_case(30 + g + K, N, d, 2)
    levels = O.build_pyramid(k, C, g)
    for t in (N - 1, 2047, 777, 5):
        trace = []
        O.select_row(qg, k, levels, t, C, g, K, True, trace)
        for rec in trace:
            assert len(rec["I"]) <= K
            assert len(rec["A"]) <= g * K


@pytest.mark.parametrize("causal", [True, False])
def test_budget_covering_every_block_selects_all(causal):
    """With K >= M_1 nothing is ever pruned: every eligible leaf is selected."""
    N, C, g, d = 999, 16, 2, 4
    qg, k = _tiny_case(40, N, d, 1)
    levels = O.build_pyramid(k, C, g)
    M1 = levels[0].shape[0]
    for t in range(0, N, 37):
        sel, gap = O.select_row(qg, k, levels, t, C, g, M1, causal)
        want = list(range(t // C + 1)) if causal else list(range(M1))
        assert sel == want and gap == math.inf


@pytest.mark.parametrize("seed,G", [(0, 1), (1, 2), (2, 4)])
def test_no_intermediate_pruning_equals_flat_lse_topk(seed, G):
    """When M_2 <= K < M_1 no intermediate level prunes, so the pyramid result is the
    forced blocks plus the best eligible leaves by exact raw-key LSE (brute force)."""
    N, C, g, d = 1024, 32, 2, 8       # M_1 = 32, M_2 = 16
    K = 16
    qg, k = _tiny_case(50 + seed, N, d, G)
    levels = O.build_pyramid(k, C, g)
    for t in range(N - 1, 0, -53):
        sel, _ = O.select_row(qg, k, levels, t, C, g, K, True)
        c = t // C
        elig = list(range(c + 1))
        if len(elig) <= K:
            assert sel == elig
            continue
        forced = {0, c, c - 1}
        free = [i for i in elig if i not in forced]
        score = np.array([sum(logsumexp(k[i * C:(i + 1) * C] @ qh / math.sqrt(d)) for qh in qg)
                          for i in free])
        order = np.lexsort((np.array(free), -score))
        want = sorted(forced | {free[j] for j in order[:K - 3]})
        assert sel == want


def test_budget_three_keeps_exactly_forced():
    """App. B with K = 3: the first, previous and current blocks and nothing else."""
    N, C, g, d = 2000, 8, 2, 4
    qg, k = _tiny_case(60, N, d, 1)
    levels = O.build_pyramid(k, C, g)
    for t in range(0, N, 13):
        c = t // C
        sel, _ = O.select_row(qg, k, levels, t, C, g, 3, True)
        assert sel == sorted({0, c} | ({c - 1} if c else set()))


def test_identical_group_heads_select_as_one_head():
    """Sec. 3.3: u is the sum of the group's head scores; G identical heads give G*s,
    which ranks exactly as one head."""
    N, C, g, K, d = 3000, 8, 2, 6, 8
    qg, k = _tiny_case(70, N, d, 1)
    levels = O.build_pyramid(k, C, g)
    for t in (N - 1, 1777, 901):
        one, _ = O.select_row(qg, k, levels, t, C, g, K, True)
        four, _ = O.select_row(np.repeat(qg, 4, axis=0), k, levels, t, C, g, K, True)
        assert one == four


def test_planted_block_wins_every_level():
    """Keys of one past block aligned with the query and every other key zero: that
    block and its ancestors carry the top score at every ranked level."""
    N, C, g, d = 4096, 16, 2, 8
    r = _rng(80)
    q = r.standard_normal((1, d))
    k = np.zeros((N, d))
    star = 100
    k[star * C:(star + 1) * C] = 25.0 * q[0] / np.linalg.norm(q[0])
    levels = O.build_pyramid(k, C, g)
    t = N - 1
    trace = []
    sel, _ = O.select_row(q, k, levels, t, C, g, 4, True, trace)
    assert star in sel
    for rec in trace:
        if rec["u"]:
            anc = star // g ** (rec["level"] - 1)
            best = max(rec["u"], key=lambda i: (rec["u"][i], -i))
            assert best == anc


# ------------------------------------------------- brute force on tiny inputs ---

def _brute_select(qg, k, t, C, g, K, causal):
    """Set-based restatement for tiny inputs: node summaries from a memoised recursive
    definition, every node's score tabulated densely, selection as set algebra."""
    N, d = k.shape
    sizes = O.level_sizes(N, C, g)
    L = len(sizes)
    memo = {}

    def summary(lv, i):
        if (lv, i) not in memo:
            if lv == 1:
                memo[(lv, i)] = k[i * C:min(i * C + C, N)].mean(0)
            else:
                kids = range(i * g, min(i * g + g, sizes[lv - 2]))
                memo[(lv, i)] = np.mean([summary(lv - 1, r) for r in kids], axis=0)
        return memo[(lv, i)]

    def kids(lv, i):
        if lv == 1:
            return k[i * C:min(i * C + C, N)]
        return np.array([summary(lv - 1, r) for r in range(i * g, min(i * g + g, sizes[lv - 2]))])

    table = {lv: np.array([sum(logsumexp(kids(lv, i) @ qh / math.sqrt(d)) for qh in qg)
                           for i in range(sizes[lv - 1])]) for lv in range(1, L + 1)}
    c = t // C
    fl = ({0, c} | ({c - 1} if c else set())) if causal else set()
    cand = {0}
    for lv in range(L, 0, -1):
        forced = {j // g ** (lv - 1) for j in fl} & cand
        if len(cand) > K:
            rest = sorted(cand - forced, key=lambda i: (-table[lv][i], i))
            cand = forced | set(rest[:K - len(forced)])
        if lv > 1:
            cand = {r for i in cand for r in range(i * g, min(i * g + g, sizes[lv - 2]))
                    if not causal or r * C * g ** (lv - 2) <= t}
    return sorted(cand)


CASES = [(N, C, g, K, G, causal, seed)
         for seed, (N, C, g, K, G, causal) in enumerate([
             (200, 2, 2, 3, 1, True), (257, 4, 2, 4, 2, True), (300, 4, 3, 5, 1, True),
             (511, 8, 4, 6, 4, True), (129, 2, 3, 7, 1, False), (100, 4, 2, 3, 2, False),
             (450, 8, 2, 8, 1, False), (333, 2, 4, 5, 2, True), (64, 2, 2, 4, 1, True),
             (480, 4, 2, 6, 1, True), (97, 8, 3, 3, 1, False), (512, 2, 2, 8, 2, True)])]


@pytest.mark.parametrize("N,C,g,K,G,causal,seed", CASES)
def test_selection_matches_brute_force(N, C, g, K, G, causal, seed):
    qg, k = _tiny_case(100 + seed, N, 4, G, scale=1.5)
    levels = O.build_pyramid(k, C, g)
    for t in sorted({0, 1, C - 1, C, N // 3, N // 2 + 1, N - 2, N - 1}):
        sel, _ = O.select_row(qg, k, levels, t, C, g, K, causal)
        assert sel == _brute_select(qg, k, t, C, g, K, causal), (t,)


# --------------------------------------------------------------- attention ---

def _sdpa(q, k, v, mask=None, causal=False):
    """torch's textbook attention in float64 on the CPU."""
    Q = torch.from_numpy(q)[None, None]
    Kt = torch.from_numpy(k)[None, None]
    V = torch.from_numpy(v)[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(Q, Kt, V, attn_mask=m, is_causal=causal)
    return o[0, 0].numpy()


@pytest.mark.parametrize("causal", [True, False])
def test_attention_with_all_blocks_is_dense_attention(causal):
    """With every block selected (K*C >= N) selected attention is dense softmax attention."""
    N, C, d = 300, 16, 8
    r = _rng(90)
    q, k, v = (r.standard_normal((N, d)) for _ in range(3))
    blocks = list(range(-(-N // C)))
    want = _sdpa(q, k, v, causal=causal)
    z = q @ k.T / math.sqrt(d)
    if causal:
        z = np.where(np.tril(np.ones((N, N), bool)), z, -np.inf)
    want_lse = logsumexp(z, axis=1)
    for t in range(0, N, 7):
        o, l = O.attention_row(q[t], k, v, blocks, t, C, causal)
        np.testing.assert_allclose(o, want[t], rtol=1e-12, atol=1e-12)
        assert l == pytest.approx(want_lse[t], rel=1e-12)


def test_attention_matches_block_masked_dense():
    """Any block set: equal to dense attention under the block (and causal) mask."""
    N, C, d, K = 256, 8, 8, 5
    r = _rng(91)
    q, k, v = (r.standard_normal((N, d)) for _ in range(3))
    M1 = N // C
    for t in range(C, N, 11):
        blocks = sorted(r.choice(t // C + 1, size=min(K, t // C + 1), replace=False))
        mask = np.zeros((1, N), bool)
        for i in blocks:
            mask[0, i * C:(i + 1) * C] = True
        mask[0, t + 1:] = False
        want = _sdpa(q[t:t + 1], k, v, mask=mask)[0]
        o, _ = O.attention_row(q[t], k, v, list(blocks) + [-1], t, C, True)
        np.testing.assert_allclose(o, want, rtol=1e-12, atol=1e-12)
    assert M1 == 32


# ---------------------------------------------------------------- flat BSA ---

@pytest.mark.parametrize("G,causal", [(1, True), (3, True), (2, False)])
def test_flat_bsa_brute_force(G, causal):
    """Sec. 3.1 + App. C.1: dense logits against every leaf mean, per-head softmax over
    the eligible non-forced blocks, head sum, top-K by lexicographic sort."""
    N, C, K, d = 1000, 8, 7, 6
    r = _rng(95 + G)
    qg = r.standard_normal((G, d))
    k = r.standard_normal((N, d))
    M1 = -(-N // C)
    S1 = np.array([k[i * C:min(i * C + C, N)].mean(0) for i in range(M1)])
    Z = qg @ S1.T / math.sqrt(d)                      # [G, M1]
    for t in range(0, N, 29):
        sel, _ = O.flat_bsa_row(qg, S1, t, C, K, causal)
        c = t // C
        elig = np.arange(M1) if not causal else np.arange(c + 1)
        if len(elig) <= K:
            assert sel == list(elig)
            continue
        forced = ({0, c} | ({c - 1} if c else set())) if causal else set()
        free = np.array([i for i in elig if i not in forced])
        u = softmax(Z[:, free], axis=1).sum(0)
        order = np.lexsort((free, -u))
        assert sel == sorted(forced | set(free[order[:K - len(forced)]].tolist()))
    # G = 1: ranking by probability equals ranking by raw score
    if G == 1:
        t = N - 1
        c = t // C
        free = [i for i in range(c + 1) if i not in {0, c, c - 1}]
        best = sorted(free, key=lambda i: (-Z[0, i], i))[:K - 3]
        assert O.flat_bsa_row(qg, S1, t, C, K, True)[0] == sorted({0, c, c - 1} | set(best))


def test_exact_ties_prefer_smaller_block_index():
    """Reading R4: bitwise-equal scores (identical key blocks, as in the needle
    workload) rank the smaller block index first, at every ranked level."""
    N, C, g, d = 2048, 16, 2, 8
    r = _rng(99)
    q = r.standard_normal((1, d))
    k = np.zeros((N, d))
    # five identical strong blocks, each in its own level-5 node (16 leaves), so every
    # ancestor path is bitwise identical; the budget leaves room for three, then two
    twins = [20, 37, 52, 70, 99]
    for b in twins:
        k[b * C:(b + 1) * C] = 10.0 * q[0] / np.linalg.norm(q[0])
    levels = O.build_pyramid(k, C, g)
    sel, gap = O.select_row(q, k, levels, N - 1, C, g, 5, True)
    c = (N - 1) // C
    assert sel == sorted({0, c - 1, c, 20, 37})
    assert gap == 0.0
    S1 = levels[0]
    sel, gap = O.flat_bsa_row(q, S1, N - 1, C, 5, True)
    assert sel == sorted({0, c - 1, c, 20, 37}) and gap == 0.0


# Decode cache (App. B): the per-token incremental rule must land on the
# direct definition of the pyramid (eq. mean_pyramid) at every length,
# including new blocks, new parents, ragged tails and a growing root.
@pytest.mark.parametrize("N,n_old,C,g", [
    (1, 0, 4, 2), (37, 0, 4, 2), (64, 1, 8, 2), (100, 31, 8, 2), (100, 32, 8, 2), (130, 63, 4, 3),
    (300, 299, 8, 4), (513, 200, 16, 2), (257, 0, 4, 2),
])
def test_pyramid_append_equals_rebuild(N, n_old, C, g):
    r = np.random.default_rng(N * 7 + n_old)
    k = r.standard_normal((N, 5))
    start = O.build_pyramid(k[:n_old], C, g) if n_old else []
    got = O.pyramid_append(start, k, n_old, C, g)
    want = O.build_pyramid(k, C, g)
    assert [x.shape for x in got] == [x.shape for x in want]
    for a, b in zip(got, want):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


def test_pyramid_append_in_steps_equals_one_append():
    r = np.random.default_rng(5)
    k = r.standard_normal((200, 3))
    lv, n = O.build_pyramid(k[:10], 8, 2), 10
    for n_new in (11, 16, 17, 63, 64, 65, 199, 200):
        lv, n = O.pyramid_append(lv, k[:n_new], n, 8, 2), n_new
    want = O.build_pyramid(k, 8, 2)
    for a, b in zip(lv, want):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)


# PISA-1 / PISA-2 (App. A "First- and second-order approximations").
def _phi(z, lam):
    """phi(lambda) = log((1/m) sum_j exp(lambda z_j)), the block's cumulant
    generating function, by its own formula (not through the oracle)."""
    return float(np.log(np.mean(np.exp(lam * np.asarray(z)))))


@pytest.mark.parametrize("seed", range(5))
def test_score_variants_are_the_cumulant_derivatives(seed):
    r = np.random.default_rng(seed)
    z = r.standard_normal(r.integers(2, 70)) * r.uniform(0.2, 3.0) + r.normal() * 2
    h = 1e-4
    d1 = (_phi(z, h) - _phi(z, -h)) / (2 * h)                 # phi'(0) = mean
    d2 = (_phi(z, h) - 2 * _phi(z, 0.0) + _phi(z, -h)) / h ** 2  # phi''(0) = population variance
    assert abs(_phi(z, 0.0)) < 1e-15
    assert abs(O.score_mean(z) - d1) < 1e-6
    assert abs((O.score_mean_var(z) - O.score_mean(z)) - 0.5 * d2) < 1e-4
    # LSE - log m = phi(1) >= phi'(0) (phi is convex): the truncations sit below it
    assert O.lse(z) - math.log(z.size) >= O.score_mean(z) - 1e-12


def test_score_variants_on_equal_logits():
    z = np.full(13, 0.625)
    assert O.score_mean(z) == 0.625 and O.score_mean_var(z) == 0.625
    assert abs(O.lse(z) - (0.625 + math.log(13))) < 1e-12


@pytest.mark.parametrize("G", [1, 3])
def test_pisa1_scores_a_node_by_its_own_summary_logit(G):
    """With the mean reducer and a mean-of-means pyramid, the mean of a node's
    child logits is the node's own logit q.S/sqrt(d) (ragged nodes included),
    so every ranked level of PISA-1 scores nodes by their own summary."""
    N, C, g, d, K = 3000, 32, 3, 8, 6
    qg, k = _tiny_case(70 + G, N, d, G)
    levels = O.build_pyramid(k, C, g)
    for t in (N - 1, 2000, 1234):
        trace = []
        O.select_row(qg, k, levels, t, C, g, K, True, trace=trace, score="mean")
        n_ranked = 0
        for lv in trace:
            for i, u in lv["u"].items():
                own = sum(float(levels[lv["level"] - 1][i] @ qh) / math.sqrt(d) for qh in qg)
                assert abs(u - own) < 1e-9 * max(1.0, abs(own))
                n_ranked += 1
        assert n_ranked > 0


@pytest.mark.parametrize("score", ["mean", "mean_var"])
def test_no_intermediate_pruning_equals_flat_topk_for_variants(score):
    """As for LSE: with M_2 <= K < M_1 the result is the forced blocks plus the
    best eligible leaves by the variant's raw-key score (brute force)."""
    N, C, g, d, K, G = 1024, 32, 2, 8, 16, 2
    qg, k = _tiny_case(91, N, d, G)
    levels = O.build_pyramid(k, C, g)

    def brute(x):
        z = x * 1.0
        m = z.mean()
        return m if score == "mean" else m + 0.5 * ((z - m) ** 2).mean()

    for t in range(N - 1, 0, -71):
        sel, _ = O.select_row(qg, k, levels, t, C, g, K, True, score=score)
        c = t // C
        elig = list(range(c + 1))
        if len(elig) <= K:
            assert sel == elig
            continue
        forced = {0, c, c - 1}
        free = [i for i in elig if i not in forced]
        sc = np.array([sum(brute(k[i * C:(i + 1) * C] @ qh / math.sqrt(d)) for qh in qg) for i in free])
        order = np.lexsort((np.array(free), -sc))
        assert sel == sorted(forced | {free[j] for j in order[:K - 3]})



# ------------------------------------------------ selection-quality diagnostic ---

@pytest.mark.parametrize("G,causal", [(1, True), (3, True), (2, False)])
def test_block_mass_is_dense_softmax_summed_per_block(G, causal):
    """App. C eq. (oracle_block_mass): exp(a(B)) / sum_B' exp(a(B')) is the
    full-attention softmax mass of B's tokens.  Checked against scipy's
    softmax over every visible token, summed per block and averaged over the
    group's heads; the masses sum to one."""
    r = _rng(11)
    N, d, C = 300, 16, 32
    k = r.standard_normal((N, d))
    qg = r.standard_normal((G, d))
    t = 250
    res = O.selection_quality_row(qg, k, [], t, C, 4, causal)
    vis = t + 1 if causal else N
    nE = -(-vis // C)
    want = np.zeros(nE)
    for h in range(G):
        p = softmax(k[:vis] @ qg[h] / math.sqrt(d))
        for b in range(nE):
            want[b] += p[b * C:min((b + 1) * C, vis)].sum() / G
    np.testing.assert_allclose(res["P"], want, rtol=1e-12, atol=1e-15)
    assert abs(res["P"].sum() - 1.0) < 1e-12
    # and a(B) itself is scipy's logsumexp over the block's visible logits
    a = O.block_log_mass(qg[0], k, t, C, causal)
    for b in range(nE):
        z = k[b * C:min((b + 1) * C, vis)] @ qg[0] / math.sqrt(d)
        assert abs(a[b] - logsumexp(z)) < 1e-12


def test_quality_of_the_reference_itself():
    """Sec. 4 eq. (oracle_metrics): a selection equal to the reference set has
    Recall@K = 1 and MassRatio = 1; its captured mass is the reference's."""
    r = _rng(12)
    N, d, C, K = 2000, 16, 32, 6
    k = r.standard_normal((N, d))
    q = r.standard_normal((2, d))
    for t in (700, 1500, 1999):
        ref = O.selection_quality_row(q, k, [], t, C, K, True)
        again = O.selection_quality_row(q, k, ref["ref"], t, C, K, True)
        assert again["recall"] == 1.0 and abs(again["ratio"] - 1.0) < 1e-12
        assert abs(again["captured"] - sum(ref["P"][b] for b in ref["ref"])) < 1e-12


def test_reference_holds_forced_and_heaviest_blocks():
    """App. C: the reference keeps the first, previous and current blocks and
    fills the rest with the eligible blocks of highest mass.  Brute force:
    rank the non-forced blocks by the dense per-block softmax mass."""
    r = _rng(13)
    N, d, C, K = 1000, 8, 20, 7
    k = r.standard_normal((N, d))
    q = r.standard_normal((1, d)) * 2.0
    t = 899
    c = t // C
    res = O.selection_quality_row(q, k, [], t, C, K, True)
    p = softmax(k[:t + 1] @ q[0] / math.sqrt(d))
    mass = np.array([p[b * C:min((b + 1) * C, t + 1)].sum() for b in range(c + 1)])
    forced = {0, c - 1, c}
    free = [b for b in np.argsort(-mass, kind="stable") if b not in forced]
    assert res["ref"] == sorted(forced | set(int(b) for b in free[:K - 3]))
    # a selection missing one reference block loses exactly that block's mass
    drop = sorted(free[:K - 3])[0]
    partial = [b for b in res["ref"] if b != drop]
    m = O.selection_quality_row(q, k, partial, t, C, K, True)
    assert abs(m["recall"] - (K - 1) / K) < 1e-15
    assert abs(m["captured"] - sum(mass[b] for b in partial)) < 1e-12
    assert abs(m["ratio"] - sum(mass[b] for b in partial) / sum(mass[b] for b in res["ref"])) < 1e-12


def test_planted_block_is_in_the_reference():
    """A block whose keys all equal a large multiple of the query carries
    nearly all the mass, so the reference (and any selection holding it)
    captures it."""
    r = _rng(14)
    N, d, C, K = 1024, 16, 32, 4
    k = r.standard_normal((N, d)) * 0.1
    q = r.standard_normal(d)
    q /= np.linalg.norm(q)
    k[10 * C:11 * C] = 40.0 * q  # logit 10 per key against ~0 elsewhere
    res = O.selection_quality_row(q[None], k, [0, 10, 30, 31], 1000, C, K, True)
    assert 10 in res["ref"] and res["captured"] > 0.99 and res["ratio"] > 0.999


def test_reference_ties_prefer_smaller_block_index():
    """Reading R15: blocks of exactly equal mass enter the reference in
    ascending index order.  Three copies of one heavy key block compete for
    two free slots (no causal policy, so nothing is forced)."""
    r = _rng(16)
    N, d, C, K = 256, 8, 32, 2
    k = r.standard_normal((N, d)) * 0.1
    q = r.standard_normal(d)
    heavy = 3.0 * q + 0.1 * r.standard_normal((C, d))
    for blk in (6, 1, 4):
        k[blk * C:(blk + 1) * C] = heavy
    res = O.selection_quality_row(q[None], k, [4, 6], N - 1, C, K, False)
    assert res["P"][1] == res["P"][4] == res["P"][6] and res["gap"] == 0.0
    assert res["ref"] == [1, 4]
    assert abs(res["recall"] - 0.5) < 1e-15


def test_all_blocks_eligible_within_budget():
    """With at most K eligible blocks the reference is all of them and holds
    all the mass; Recall@K divides by K (reading R15)."""
    r = _rng(15)
    k = r.standard_normal((200, 8))
    q = r.standard_normal((1, 8))
    res = O.selection_quality_row(q, k, [0, 1, 2], 100, 32, 8, True)
    assert res["ref"] == [0, 1, 2, 3]
    assert abs(res["recall"] - 3 / 8) < 1e-15
    assert abs(sum(res["P"][b] for b in res["ref"]) - 1.0) < 1e-12


# -------------------------------------------------- backward, indices fixed ---

def _masked_dense_grads(q, k, v, idx, do, C, causal):
    """torch float64 autograd through dense attention with a block mask built
    from the selected indices (the library's own softmax and matmul)."""
    B, H, Nq, d = q.shape
    Hkv, N = k.shape[1], k.shape[2]
    G = H // Hkv
    qt = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    kt = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    mask = torch.zeros((B, Hkv, Nq, N), dtype=torch.bool)
    for b in range(B):
        for h in range(Hkv):
            for r in range(Nq):
                t = N - Nq + r
                for blk in idx[b, h, r]:
                    if blk < 0:
                        continue
                    hi = min((blk + 1) * C, N)
                    if causal:
                        hi = min(hi, t + 1)
                    mask[b, h, r, blk * C:hi] = True
    kx = kt.repeat_interleave(G, dim=1)
    vx = vt.repeat_interleave(G, dim=1)
    z = qt @ kx.transpose(-1, -2) / math.sqrt(d)
    z = z.masked_fill(~mask.repeat_interleave(G, dim=1), float("-inf"))
    o = torch.softmax(z, dim=-1) @ vx
    (o * torch.tensor(do, dtype=torch.float64)).sum().backward()
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


@pytest.mark.parametrize("G,causal", [(1, True), (2, True), (3, False)])
def test_backward_equals_autograd_of_block_masked_attention(G, causal):
    """App. B (indices held fixed): the oracle's gradients equal torch's
    autograd of dense attention restricted to the selected tokens."""
    r = _rng(21)
    B, Hkv, Nq, N, d, C, K = 1, 2, 70, 200, 16, 16, 4
    H = Hkv * G
    q = r.standard_normal((B, H, Nq, d))
    k = r.standard_normal((B, Hkv, N, d))
    v = r.standard_normal((B, Hkv, N, d))
    do = r.standard_normal((B, H, Nq, d))
    M1 = -(-N // C)
    idx = np.full((B, Hkv, Nq, K), -1)
    for h in range(Hkv):
        for row in range(Nq):
            t = N - Nq + row
            top = t // C if causal else M1 - 1
            pick = sorted(r.choice(top + 1, size=min(K, top + 1), replace=False))
            idx[0, h, row, :len(pick)] = pick
    got = O.sparse_attention_bwd(q, k, v, idx, do, C, causal)
    want = _masked_dense_grads(q, k, v, idx, do, C, causal)
    for g_, w_ in zip(got, want):
        np.testing.assert_allclose(g_, w_, rtol=1e-10, atol=1e-12)


def test_backward_matches_finite_differences():
    """The gradient of L = sum(do * o) by central differences of the oracle's
    own forward (attention_row), one coordinate of q, k and v at a time."""
    r = _rng(22)
    N, d, C, t = 40, 6, 8, 33
    q = r.standard_normal(d)
    k = r.standard_normal((N, d))
    v = r.standard_normal((N, d))
    do = r.standard_normal(d)
    blocks = [0, 2, 3, 4]

    def loss(qq, kk, vv):
        return float(O.attention_row(qq, kk, vv, blocks, t, C, True)[0] @ do)

    dq, tok, dk, dv = O.attention_row_bwd(q, k, v, blocks, t, C, True, do)
    eps = 1e-6
    for i in range(d):
        e = np.zeros(d)
        e[i] = eps
        assert abs((loss(q + e, k, v) - loss(q - e, k, v)) / (2 * eps) - dq[i]) < 1e-7
    for j, tj in enumerate(tok[::5]):
        for i in (0, d - 1):
            kp, km = k.copy(), k.copy()
            kp[tj, i] += eps
            km[tj, i] -= eps
            assert abs((loss(q, kp, v) - loss(q, km, v)) / (2 * eps) - dk[tok.index(tj), i]) < 1e-7
            vp, vm = v.copy(), v.copy()
            vp[tj, i] += eps
            vm[tj, i] -= eps
            assert abs((loss(q, k, vp) - loss(q, k, vm)) / (2 * eps) - dv[tok.index(tj), i]) < 1e-7
    # a token outside the selection (block 1) and a future token get no gradient
    assert 9 not in tok and 35 not in tok


def test_attention_ignores_blocks_past_the_end():
    """Blocks at or past ceil(N/C) hold no tokens, whatever the index type
    (int32 arrays included: block * C must not wrap)."""
    r = _rng(41)
    N, C, d = 300, 16, 8
    q, k, v = r.standard_normal(d), r.standard_normal((N, d)), r.standard_normal((N, d))
    base = np.array([0, 3, 7, 18], dtype=np.int32)
    want = O.attention_row(q, k, v, base, N - 1, C, True)
    for extra in (19, 25, (1 << 30) - 1, (1 << 31) - 1):
        got = O.attention_row(q, k, v, np.append(base, np.int32(extra)), N - 1, C, True)
        assert np.array_equal(got[0], want[0]) and got[1] == want[1], extra
        gb = O.attention_row_bwd(q, k, v, np.append(base, np.int32(extra)), N - 1, C, True, r.standard_normal(d))
        assert all(0 <= j < N for j in gb[1])
