"""CPU oracle for PISA's data-parallel hot path -- TEST INFRASTRUCTURE ONLY.

This is a plain, slow, float64 restatement of what the paper defines, used to
check the HIP library.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import it; the product path never does.
It shares no code with the HIP library and imports nothing from the package.

Paper: "Block Sparse Attention with Log-Linear Complexity" (PISA).
Indices are 0-based here (the paper counts from 1).  All arithmetic is
float64; bf16 inputs widen to float64 exactly.

Contents and the passage each follows:

* ``level_sizes``       -- hierarchy sizes, Sec. 3.2 eq. (key_hierarchy):
                           M_1 = ceil(N/C), M_{l+1} = ceil(M_l / g).
* ``build_pyramid``     -- mean pyramid, Sec. 3.2 eq. (mean_pyramid): leaf
                           means of raw keys, then means over the *valid*
                           children one level down.
* ``pyramid_append``    -- decode-cache update, App. B ("Decode cache"):
                           per token, the running mean of its leaf and the
                           ancestor path (pinned against build_pyramid).
* ``lse``               -- natural-log LogSumExp, max-subtracted.
* ``score_mean``, ``score_mean_var`` -- the PISA-1 / PISA-2 block scores,
                           App. A "First- and second-order approximations".
* ``select_row``        -- coarse-to-fine Top-K, Sec. 3.2 eq.
                           (hierarchical_topk) with the LSE score of eq.
                           (direct_child_lse), the grouped-head sum of
                           Sec. 3.3 eq. (kernel_grouped_score) and the causal
                           eligibility / forced-block policy of App. B.
* ``attention_row``     -- selected sparse attention, Sec. 3.1 eq.
                           (selected_sparse_attention), causal cut of App. B.
* ``flat_bsa_row``      -- flat block selection, Sec. 3.1 eqs.
                           (bsa_block_scores, bsa_topk), with the per-head
                           normalisation before the head sum of App. C.1.
* ``attention_row_bwd`` -- backward of the selected sparse attention with
                           the selection held fixed (App. B: the backward
                           pass treats the chosen block indices as
                           constants): the gradients of eq.
                           (selected_sparse_attention) with respect to q, k, v
                           over the selected, visible tokens only.
* ``block_log_mass``, ``selection_quality_row`` -- the block-selection
                           diagnostic of Sec. 4 ("Block-selection quality",
                           eq. oracle_metrics) and App. C ("Block-selection
                           diagnostic", eq. oracle_block_mass): per-block
                           log mass of the full attention, the head-averaged
                           block mass P, the full-attention reference set and
                           Recall@K / CapturedMass / MassRatio of a selection.

Readings of points the paper leaves open (each also recorded in the design
notes of the repository):

* R1  levels: the root sits at level L (M_L = 1) and is never scored.
* R2  forced set: in causal mode the first, previous and current leaf blocks
      and all their ancestors are kept inside the K budget without scores;
      causal mode needs K >= 3.
* R3  the "at most K candidates" test counts every eligible candidate,
      forced ones included.
* R4  ties: higher score first, then the smaller block index.
* R5  eligibility: node i of level l (covering tokens from i*C*g^(l-1)) is a
      candidate only if it exists and, in causal mode, starts at or before t.
* R6  query row i sits at absolute position t = N - Nq + i.
* R7  flat-BSA head normalisation = softmax over the eligible non-forced
      blocks of each head, then the sum over the group's heads.
* R8  grouped-query heads: query head h' uses KV head h' // (H / Hkv).
* R9  outputs: selected leaf indices ascending, padded with -1 to K.
* R10 attention with no visible token returns o = 0 and lse = -inf.
* R15 diagnostic reference set: the forced blocks of R2 plus the eligible
      blocks of highest grouped mass P, ties to the smaller index (R4); with
      at most K eligible blocks it is all of them.  Recall@K divides by K as
      printed, also for rows with fewer than K eligible blocks.
"""
from __future__ import annotations

import math

import numpy as np

NEG_INF = -math.inf
POS_INF = math.inf


def level_sizes(N: int, C: int, g: int) -> list[int]:
    """Return [M_1, ..., M_L] of the key hierarchy (Sec. 3.2, eq. key_hierarchy).

    M_1 = ceil(N / C) leaf blocks; each coarser level merges up to g adjacent
    blocks, M_{l+1} = ceil(M_l / g), until a single root block remains.
    """
    if N < 1 or C < 1 or g < 2:
        raise ValueError("need N >= 1, C >= 1, g >= 2")
    sizes = [-(-N // C)]
    while sizes[-1] > 1:
        sizes.append(-(-sizes[-1] // g))
    return sizes


def build_pyramid(k: np.ndarray, C: int, g: int) -> list[np.ndarray]:
    """Mean pyramid of one KV head (Sec. 3.2, eq. mean_pyramid).

    k: [N, d] keys.  Returns a list whose entry l-1 is the [M_l, d] array of
    level-l summaries, l = 1..L.  Level 1 is the mean of the raw keys of each
    leaf block (the last block may hold fewer than C keys); level l+1 is the
    mean of the existing children at level l (the denominator counts valid
    children only).
    """
    k = np.asarray(k, dtype=np.float64)
    N, d = k.shape
    M = level_sizes(N, C, g)
    levels = []
    leaf = np.empty((M[0], d))
    for i in range(M[0]):
        leaf[i] = k[i * C:min((i + 1) * C, N)].mean(axis=0)
    levels.append(leaf)
    for lv in range(1, len(M)):
        below = levels[-1]
        cur = np.empty((M[lv], d))
        for i in range(M[lv]):
            cur[i] = below[i * g:min((i + 1) * g, M[lv - 1])].mean(axis=0)
        levels.append(cur)
    return levels


def pyramid_append(levels: list[np.ndarray], k: np.ndarray, n_old: int, C: int, g: int) -> list[np.ndarray]:
    """Decode-cache update (App. B, paragraph "Decode cache"): extend the
    pyramid of the first n_old keys (``levels`` as from build_pyramid; an
    empty list when n_old = 0) to all len(k) keys, one token at a time.

    A new token moves the running mean of its leaf block (or opens a new
    block).  Going up, a parent is the mean of its existing children: when one
    child moves by delta the parent moves by delta / (number of children);
    when a child is new the parent becomes prev + (child - prev) / n; a parent
    that did not exist is created from its first child; and when the top
    level gains a second node a new root (the mean of the top level) is
    added.  Returns the new list of levels (same form as build_pyramid).
    """
    k = np.asarray(k, dtype=np.float64)
    rows = [[r.copy() for r in lv] for lv in levels] or [[]]
    for t in range(n_old, k.shape[0]):
        c, cnt = divmod(t, C)
        leaf = rows[0]
        if cnt == 0:
            leaf.append(k[t].copy())
            before = None
        else:
            before = leaf[c].copy()
            leaf[c] = before + (k[t] - before) / (cnt + 1)
        child, lv = c, 0
        while True:
            cur = rows[lv]
            if lv == len(rows) - 1:          # the top level
                if len(cur) > 1:             # it outgrew the root: one level more
                    rows.append([np.mean(np.array(cur[:g]), axis=0)])
                break
            parent = child // g
            n_children = min(g, len(cur) - parent * g)
            up = rows[lv + 1]
            if parent == len(up):            # first child of a new parent
                up.append(cur[child].copy())
                before = None
            else:
                prev = up[parent].copy()
                if before is None:           # one child more in the mean
                    up[parent] = prev + (cur[child] - prev) / n_children
                else:                        # the child's share moved
                    up[parent] = prev + (cur[child] - before) / n_children
                before = prev
            child, lv = parent, lv + 1
    return [np.array(lv) for lv in rows]


def lse(z: np.ndarray) -> float:
    """Natural-log LogSumExp of a 1-D array, max-subtracted."""
    z = np.asarray(z, dtype=np.float64)
    if z.size == 0:
        return NEG_INF
    m = float(z.max())
    if m == NEG_INF:
        return NEG_INF
    return m + math.log(float(np.exp(z - m).sum()))


def score_mean(z: np.ndarray) -> float:
    """PISA-1 block score (App. A, first-order truncation): the mean logit."""
    z = np.asarray(z, dtype=np.float64)
    return float(z.sum() / z.size)


def score_mean_var(z: np.ndarray) -> float:
    """PISA-2 block score (App. A, second-order truncation): the mean logit
    plus half the population variance (denominator m)."""
    z = np.asarray(z, dtype=np.float64)
    mean = z.sum() / z.size
    return float(mean + 0.5 * ((z - mean) ** 2).sum() / z.size)


SCORES = {"lse": lse, "mean": score_mean, "mean_var": score_mean_var}


def forced_leaves(t: int, C: int, causal: bool) -> set[int]:
    """First, previous and current leaf block of position t (App. B); empty if not causal."""
    if not causal:
        return set()
    c = t // C
    f = {0, c}
    if c >= 1:
        f.add(c - 1)
    return f


def select_row(qg: np.ndarray, k: np.ndarray, levels: list[np.ndarray], t: int,
               C: int, g: int, K: int, causal: bool, trace: list | None = None, score: str = "lse"):
    """Pyramid Top-K selection for one query position and one KV head.

    qg: [G, d] the query vectors of the G heads that share this KV head.
    k:  [N, d] raw keys of the KV head (leaf-level scoring reads them).
    levels: output of ``build_pyramid`` for the same keys.
    t: absolute position of the query.

    Returns (selected leaf indices ascending, min_gap) where min_gap is the
    smallest margin, over all ranked levels, between the lowest kept score
    and the highest dropped score (+inf if no level needed ranking).  If
    ``trace`` is a list, one dict per level is appended with the candidate
    set A, forced set F, kept set I and the scores u.  ``score`` names the
    per-head block score: "lse" (PISA), "mean" (PISA-1) or "mean_var"
    (PISA-2, App. A); the group's per-head scores are summed in every case.

    Steps (Sec. 3.2 eq. hierarchical_topk, eq. direct_child_lse; Sec. 3.3
    eq. kernel_grouped_score; App. B):
      start with the root at level L; at each level l = L..1 keep every
      candidate if there are at most K of them, otherwise score each
      non-forced candidate by the sum over the G heads of the LSE of its
      children's scaled logits (child summaries of level l-1, or the raw keys
      of the leaf block when l = 1) and keep the forced candidates plus the
      K - |F| best scored ones; expand the kept blocks to their eligible
      children at level l-1.
    """
    qg = np.asarray(qg, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    N, d = k.shape
    M = [lv.shape[0] for lv in levels]
    L = len(M)
    scale = 1.0 / math.sqrt(d)
    f_leaf = forced_leaves(t, C, causal)
    reduce = SCORES[score]

    def span(lv: int) -> int:
        return C * g ** (lv - 1)

    def eligible(lv: int, i: int) -> bool:
        return i < M[lv - 1] and (not causal or i * span(lv) <= t)

    def children(lv: int, i: int) -> range:
        return range(i * g, min((i + 1) * g, M[lv - 2]))

    A = [0]
    min_gap = POS_INF
    I: list[int] = [0]
    for lv in range(L, 0, -1):
        F = {j // g ** (lv - 1) for j in f_leaf} & set(A)
        u: dict[int, float] = {}
        if len(A) <= K:
            I = sorted(A)
        else:
            free = [i for i in A if i not in F]
            for i in free:
                if lv >= 2:
                    x = levels[lv - 2][list(children(lv, i))]
                else:
                    x = k[i * C:min((i + 1) * C, N)]
                u[i] = sum(reduce(x @ qh * scale) for qh in qg)
            ranked = sorted(free, key=lambda i: (-u[i], i))
            n_keep = K - len(F)
            keep, drop = ranked[:n_keep], ranked[n_keep:]
            if keep and drop:
                min_gap = min(min_gap, u[keep[-1]] - u[drop[0]])
            I = sorted(F | set(keep))
        if trace is not None:
            trace.append({"level": lv, "A": list(A), "F": set(F), "I": list(I), "u": dict(u)})
        if lv > 1:
            A = [r for i in I for r in children(lv, i) if eligible(lv - 1, r)]
    return I, min_gap


def candidate_score(qg: np.ndarray, k: np.ndarray, levels: list[np.ndarray], lv: int, i: int,
                    C: int, g: int, score: str = "lse") -> float:
    """Grouped score u of node i at level lv >= 1 for the query heads qg [G, d]
    (Sec. 3.2 eq. direct_child_lse, summed over heads by Sec. 3.3 eq.
    kernel_grouped_score): the sum over the heads of the reducer of the
    children's scaled logits -- the summaries of level lv-1 for lv >= 2, the
    raw keys of leaf block i for lv = 1.  Same per-candidate arithmetic as
    ``select_row`` (so equal inputs give bit-equal scores)."""
    qg = np.asarray(qg, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    N, d = k.shape
    scale = 1.0 / math.sqrt(d)
    if lv >= 2:
        below = levels[lv - 2]
        x = below[list(range(i * g, min((i + 1) * g, below.shape[0])))]
    else:
        x = k[i * C:min((i + 1) * C, N)]
    reduce = SCORES[score]
    return sum(reduce(x @ qh * scale) for qh in qg)


def _kept_set_ok(kept, u: dict, tol: float, strict_ties: bool) -> bool:
    """A kept subset of the scored candidates is admissible when no dropped
    candidate beats a kept one by more than tol; with strict_ties a kept and a
    dropped candidate of exactly equal score must follow the tie rule R4
    (the smaller index is kept)."""
    kept = set(kept)
    ks = [u[i] for i in kept]
    ds = [u[j] for j in u if j not in kept]
    if not ks or not ds:
        return True
    if min(ks) < max(ds) - tol:
        return False
    if strict_ties:
        for i in kept:
            for j in u:
                if j not in kept and u[j] == u[i] and j < i:
                    return False
    return True


def selection_admissible(qg: np.ndarray, k: np.ndarray, levels: list[np.ndarray], t: int, C: int, g: int,
                         K: int, causal: bool, chosen, tol: float = 1e-3, score: str = "lse",
                         strict_ties: bool = True, budget: int = 4000) -> dict:
    """Is the leaf set ``chosen`` a possible outcome of the coarse-to-fine
    selection of ``select_row`` when every ranking may be decided by scores
    that differ from the exact ones by rounding (a kept candidate may score up
    to ``tol`` below a dropped one)?

    A selector that computes every score within tol/2 of the exact value and
    otherwise follows Sec. 3.2 eq. hierarchical_topk (with the App. B forced
    set and eligibility) produces an admissible set; on rows whose exact
    margins all exceed tol the only admissible set is ``select_row``'s.

    The replay walks the levels from the root.  At each level the kept set
    must contain the ancestors of every chosen leaf (a leaf is a candidate only
    below kept ancestors), keep the forced nodes, and be admissible in the
    sense of ``_kept_set_ok``; the remaining slots may be filled by any
    admissible choice, which changes the next level's candidates, so the
    choices are searched depth first (exact ranking first, then the other
    admissible fills of the tie band).  At the leaf level the kept set is
    ``chosen`` itself.

    Returns a dict: ``ok`` (True / False, or None when ``budget`` level visits
    did not settle it), ``leaf_ranked`` (whether the accepted path ranked the
    leaf level, i.e. whether the chosen blocks carry scores), ``leaf_u`` (the
    exact leaf scores of the accepted path's scored candidates), ``visits``.
    """
    qg = np.asarray(qg, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    N, d = k.shape
    M = [lv.shape[0] for lv in levels]
    L = len(M)
    f_leaf = forced_leaves(t, C, causal)
    chosen = {int(j) for j in chosen if j >= 0}

    def span(lv: int) -> int:
        return C * g ** (lv - 1)

    def eligible(lv: int, i: int) -> bool:
        return i < M[lv - 1] and (not causal or i * span(lv) <= t)

    def children(lv: int, i: int) -> range:
        return range(i * g, min((i + 1) * g, M[lv - 2]))

    need = {lv: {j // g ** (lv - 1) for j in chosen} for lv in range(1, L + 1)}
    state = {"visits": 0, "leaf_ranked": False, "leaf_u": {}}
    dead: set = set()

    class _Budget(Exception):
        pass

    def fills(free, u, n_keep, must):
        """Admissible kept sets of size n_keep that contain ``must``, the exact
        ranking's first."""
        if n_keep == 0:
            if not must:
                yield set()
            return
        ranked = sorted(free, key=lambda i: (-u[i], i))
        hi, lo = u[ranked[n_keep - 1]], u[ranked[n_keep]]
        sure = [i for i in ranked if u[i] > hi + tol]
        band = [i for i in ranked if lo - tol <= u[i] <= hi + tol]
        if not must <= set(sure) | set(band):
            return
        fixed = set(sure) | (must & set(band))
        rest = [i for i in band if i not in fixed]
        r = n_keep - len(fixed)
        if r < 0 or r > len(rest):
            return
        from itertools import combinations
        for extra in combinations(rest, r):
            S = fixed | set(extra)
            if _kept_set_ok(S, u, tol, strict_ties):
                yield S

    def visit(lv: int, A: list) -> bool:
        state["visits"] += 1
        if state["visits"] > budget:
            raise _Budget()
        key = (lv, tuple(sorted(A)))
        if key in dead:
            return False
        A_set = set(A)
        if not need[lv] <= A_set:
            dead.add(key)
            return False
        F = {j // g ** (lv - 1) for j in f_leaf} & A_set
        if len(A) <= K:
            options = [A_set]
            u = {}
        else:
            free = [i for i in A if i not in F]
            u = {i: candidate_score(qg, k, levels, lv, i, C, g, score) for i in free}
            n_keep = K - len(F)
            if lv == 1:
                S = chosen - F
                ok_leaf = (F <= chosen and len(S) == n_keep and S <= set(free)
                           and _kept_set_ok(S, u, tol, strict_ties))
                options = [chosen] if ok_leaf else []
            else:
                options = (F | S for S in fills(free, u, n_keep, need[lv] - F))
        for I in options:
            if lv == 1:
                if set(I) == chosen:
                    state["leaf_ranked"] = len(A) > K
                    state["leaf_u"] = dict(u)
                    return True
                continue
            nxt = [r for i in sorted(I) for r in children(lv, i) if eligible(lv - 1, r)]
            if visit(lv - 1, nxt):
                return True
        dead.add(key)
        return False

    try:
        ok = visit(L, [0])
    except _Budget:
        ok = None
    return {"ok": ok, "leaf_ranked": state["leaf_ranked"], "leaf_u": state["leaf_u"], "visits": state["visits"]}


def flat_bsa_admissible(qg: np.ndarray, leaf_means: np.ndarray, t: int, C: int, K: int, causal: bool,
                        chosen, tol: float = 1e-3, strict_ties: bool = True) -> bool:
    """Is ``chosen`` a possible flat-BSA selection (``flat_bsa_row``) under
    rounding of the scores by up to tol (log units of the summed per-head
    probabilities)?  The forced blocks must be kept and no dropped eligible
    block may beat a kept one by more than tol."""
    qg = np.asarray(qg, dtype=np.float64)
    S1 = np.asarray(leaf_means, dtype=np.float64)
    M1, d = S1.shape
    c = t // C
    E = [i for i in range(M1) if not causal or i <= c]
    chosen = {int(j) for j in chosen if j >= 0}
    if len(E) <= K:
        return chosen == set(E)
    F = forced_leaves(t, C, causal) & set(E)
    free = [i for i in E if i not in F]
    z = qg @ S1[free].T / math.sqrt(d)
    p = np.zeros(len(free))
    for zh in z:
        p += np.exp(zh - lse(zh))
    u = dict(zip(free, np.log(p)))
    S = chosen - F
    return F <= chosen and len(S) == K - len(F) and S <= set(free) and _kept_set_ok(S, u, tol, strict_ties)


def attention_row(q: np.ndarray, k: np.ndarray, v: np.ndarray, blocks, t: int,
                  C: int, causal: bool):
    """Attention of one query over the tokens of the selected leaf blocks.

    Sec. 3.1 eq. (selected_sparse_attention): softmax of q.k_j / sqrt(d) over
    the union of the selected blocks' tokens, weights applied to the original
    values; App. B: tokens after t are masked in causal mode.
    Returns (o [d], lse) with lse the natural-log normaliser of the scaled
    logits.  Negative block indices are padding and ignored.
    """
    q = np.asarray(q, dtype=np.float64)
    N, d = k.shape
    tokens = sorted({j for i in map(int, blocks) if i >= 0
                     for j in range(i * C, min((i + 1) * C, N))
                     if not causal or j <= t})
    if not tokens:
        return np.zeros(d), NEG_INF
    kk = np.asarray(k[tokens], dtype=np.float64)
    vv = np.asarray(v[tokens], dtype=np.float64)
    z = kk @ q / math.sqrt(d)
    row_lse = lse(z)
    p = np.exp(z - row_lse)
    return p @ vv, row_lse


def attention_row_bwd(q: np.ndarray, k: np.ndarray, v: np.ndarray, blocks, t: int, C: int, causal: bool,
                      do: np.ndarray):
    """Gradients of one query's selected attention (App. B: indices fixed).

    With z_j = q.k_j / sqrt(d) over the selected visible tokens T, p = softmax(z),
    o = sum_j p_j v_j and the output gradient do:
        dv_j = p_j do,   dp_j = do.v_j,   D = do.o,   ds_j = p_j (dp_j - D),
        dq = sum_j ds_j k_j / sqrt(d),   dk_j = ds_j q / sqrt(d).
    Returns (dq [d], tokens [|T|], dk [|T|, d], dv [|T|, d]): the per-token
    contributions, to be summed over every query row and head that reaches
    the token.
    """
    q = np.asarray(q, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    N, d = k.shape
    tokens = sorted({j for i in map(int, blocks) if i >= 0
                     for j in range(i * C, min((i + 1) * C, N))
                     if not causal or j <= t})
    if not tokens:
        return np.zeros(d), [], np.zeros((0, d)), np.zeros((0, d))
    kk = np.asarray(k[tokens], dtype=np.float64)
    vv = np.asarray(v[tokens], dtype=np.float64)
    z = kk @ q / math.sqrt(d)
    p = np.exp(z - lse(z))
    o = p @ vv
    dv = p[:, None] * do[None, :]
    dp = vv @ do
    ds = p * (dp - float(do @ o))
    dq = ds @ kk / math.sqrt(d)
    dk = ds[:, None] * q[None, :] / math.sqrt(d)
    return dq, tokens, dk, dv


def flat_bsa_row(qg: np.ndarray, leaf_means: np.ndarray, t: int, C: int, K: int,
                 causal: bool):
    """Flat (single-level) block selection for one position and KV head.

    Sec. 3.1: score every eligible leaf summary, s_i = q.kbar_i / sqrt(d)
    (eq. bsa_block_scores), keep the K best (eq. bsa_topk).  App. C.1: the
    scores are normalised within each query head before the sum over heads
    (reading R7: softmax over the eligible non-forced blocks).  The forced
    blocks of App. B are kept inside the budget.

    Returns (selected indices ascending, min_gap) with the gap measured in
    log units of the summed probabilities (equal to logit units when G = 1).
    """
    qg = np.asarray(qg, dtype=np.float64)
    S1 = np.asarray(leaf_means, dtype=np.float64)
    M1, d = S1.shape
    c = t // C
    E = [i for i in range(M1) if not causal or i <= c]
    if len(E) <= K:
        return sorted(E), POS_INF
    F = forced_leaves(t, C, causal) & set(E)
    free = [i for i in E if i not in F]
    z = qg @ S1[free].T / math.sqrt(d)          # [G, |free|]
    u = np.zeros(len(free))
    for zh in z:
        u += np.exp(zh - lse(zh))
    logu = np.log(u)
    order = sorted(range(len(free)), key=lambda j: (-logu[j], free[j]))
    n_keep = K - len(F)
    keep = [free[j] for j in order[:n_keep]]
    gap = POS_INF
    if n_keep > 0 and n_keep < len(free):
        gap = logu[order[n_keep - 1]] - logu[order[n_keep]]
    return sorted(F | set(keep)), gap


def block_log_mass(q: np.ndarray, k: np.ndarray, t: int, C: int, causal: bool) -> np.ndarray:
    """Log mass of every eligible leaf block for one query vector (App. C,
    eq. oracle_block_mass): a(B) = log sum over the tokens j of B (j <= t
    when causal) of exp(q.k_j / sqrt(d)).  Returns an array over the blocks
    0 .. |E|-1 (E = the causally available blocks, all blocks if not causal).
    """
    q = np.asarray(q, dtype=np.float64)
    N, d = k.shape
    M1 = -(-N // C)
    nE = min(t // C + 1, M1) if causal else M1
    a = np.empty(nE)
    for b in range(nE):
        hi = min((b + 1) * C, N)
        if causal:
            hi = min(hi, t + 1)
        z = np.asarray(k[b * C:hi], dtype=np.float64) @ q / math.sqrt(d)
        a[b] = lse(z)
    return a


def selection_quality_row(qg: np.ndarray, k: np.ndarray, sel, t: int, C: int, K: int, causal: bool):
    """Selection quality of one (query position, KV head) against the
    full-attention reference (Sec. 4 eq. oracle_metrics; App. C).

    qg: [G, d] queries of the KV head's query heads; sel: selected leaf
    blocks (negative entries are padding).  P(B) is, for each head, the
    softmax of the block log masses over the eligible blocks, averaged over
    the G heads.  The reference set holds the forced blocks (App. B) and
    fills the remaining budget with the eligible blocks of highest P.

    Returns a dict: recall = |sel & ref| / K, captured = sum of P over sel,
    ratio = captured / (sum of P over ref), ref (ascending list), P (array
    over the eligible blocks), gap (smallest kept minus largest dropped P
    among the ranked blocks, +inf if nothing was ranked).
    """
    qg = np.asarray(qg, dtype=np.float64)
    G = qg.shape[0]
    P = None
    for h in range(G):
        a = block_log_mass(qg[h], k, t, C, causal)
        ph = np.exp(a - lse(a))
        P = ph if P is None else P + ph
    P = P / G
    nE = P.size
    E = list(range(nE))
    gap = POS_INF
    if nE <= K:
        ref = E
    else:
        F = forced_leaves(t, C, causal) & set(E)
        free = [b for b in E if b not in F]
        order = sorted(free, key=lambda b: (-P[b], b))
        n_keep = K - len(F)
        ref = sorted(F | set(order[:n_keep]))
        if 0 < n_keep < len(free):
            gap = P[order[n_keep - 1]] - P[order[n_keep]]
    chosen = sorted({int(b) for b in sel if b >= 0})
    captured = float(sum(P[b] for b in chosen if b < nE))
    ref_mass = float(sum(P[b] for b in ref))
    return {"recall": len(set(chosen) & set(ref)) / K, "captured": captured,
            "ratio": captured / ref_mass if ref_mass > 0 else 0.0, "ref": ref, "P": P, "gap": gap}


# ---------------------------------------------------------------------------
# Whole-tensor drivers (loops over batch, heads and the requested rows).
# ---------------------------------------------------------------------------

def pyramid_rows(levels: list[np.ndarray]) -> np.ndarray:
    """Concatenate levels 1..max(1, L-1) (the root is never scored) into [R, d]."""
    keep = levels[:-1] if len(levels) > 1 else levels
    return np.concatenate(keep, axis=0)


def _group(H: int, Hkv: int) -> int:
    if H % Hkv:
        raise ValueError("H must be a multiple of Hkv")
    return H // Hkv


def pyramid(k: np.ndarray, C: int, g: int) -> np.ndarray:
    """[B, Hkv, N, d] keys -> [B, Hkv, R, d] concatenated pyramid (float64)."""
    B, Hkv, N, d = k.shape
    out = None
    for b in range(B):
        for h in range(Hkv):
            rows = pyramid_rows(build_pyramid(k[b, h], C, g))
            if out is None:
                out = np.empty((B, Hkv, rows.shape[0], d))
            out[b, h] = rows
    return out


def select(q, k, C, g, K, causal, rows=None, heads=None, score="lse"):
    """Selection for rows of every (batch, KV head).

    q: [B, H, Nq, d], k: [B, Hkv, N, d].  rows: iterable of query-row indices
    (default all).  Returns (idx [B, Hkv, len(rows), K] int64 padded with -1,
    gap [B, Hkv, len(rows)]).
    """
    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = _group(H, Hkv)
    rows = list(range(Nq)) if rows is None else list(rows)
    heads = list(range(Hkv)) if heads is None else list(heads)
    idx = np.full((B, len(heads), len(rows), K), -1, dtype=np.int64)
    gap = np.full((B, len(heads), len(rows)), POS_INF)
    for b in range(B):
        for hi, h in enumerate(heads):
            kh = np.asarray(k[b, h], dtype=np.float64)
            levels = build_pyramid(kh, C, g)
            for ri, r in enumerate(rows):
                t = N - Nq + r
                qg = q[b, h * G:(h + 1) * G, r]
                sel, gp = select_row(qg, kh, levels, t, C, g, K, causal, score=score)
                idx[b, hi, ri, :len(sel)] = sel
                gap[b, hi, ri] = gp
    return idx, gap


def sparse_attention(q, k, v, block_idx, C, causal, rows=None, heads=None):
    """Attention for rows of every query head given selected blocks.

    block_idx: [B, Hkv, Nq_or_len(rows), K] (indexed by position in ``rows``
    when ``rows`` is given).  Returns (o [B, Hsel, len(rows), d],
    lse [B, Hsel, len(rows)]) where Hsel enumerates ``heads`` (query heads,
    default all).
    """
    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = _group(H, Hkv)
    rows = list(range(Nq)) if rows is None else list(rows)
    heads = list(range(H)) if heads is None else list(heads)
    o = np.zeros((B, len(heads), len(rows), d))
    out_lse = np.zeros((B, len(heads), len(rows)))
    for b in range(B):
        for hi, hq in enumerate(heads):
            hk = hq // G
            for ri, r in enumerate(rows):
                t = N - Nq + r
                o[b, hi, ri], out_lse[b, hi, ri] = attention_row(
                    q[b, hq, r], k[b, hk], v[b, hk], block_idx[b, hk, ri], t, C, causal)
    return o, out_lse


def select_flat_bsa(q, k, C, K, causal, rows=None, heads=None):
    """Flat-BSA selection for rows of every (batch, KV head); same layout as ``select``."""
    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = _group(H, Hkv)
    rows = list(range(Nq)) if rows is None else list(rows)
    heads = list(range(Hkv)) if heads is None else list(heads)
    idx = np.full((B, len(heads), len(rows), K), -1, dtype=np.int64)
    gap = np.full((B, len(heads), len(rows)), POS_INF)
    for b in range(B):
        for hi, h in enumerate(heads):
            S1 = build_pyramid(np.asarray(k[b, h], dtype=np.float64), C, 2)[0]
            for ri, r in enumerate(rows):
                t = N - Nq + r
                sel, gp = flat_bsa_row(q[b, h * G:(h + 1) * G, r], S1, t, C, K, causal)
                idx[b, hi, ri, :len(sel)] = sel
                gap[b, hi, ri] = gp
    return idx, gap


def selection_quality(q, k, block_idx, C, K, causal, rows, heads=None):
    """Diagnostic for the given rows of every (batch, KV head).

    block_idx: [B, Hkv, len(rows), K] selections of those rows.  Returns
    (metrics [B, Hkv, len(rows), 3] = recall, captured, ratio;
    ref [B, Hkv, len(rows), K] ascending, -1 padded; gap [B, Hkv, len(rows)]).
    """
    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = _group(H, Hkv)
    rows = list(rows)
    heads = list(range(Hkv)) if heads is None else list(heads)
    met = np.zeros((B, len(heads), len(rows), 3))
    ref = np.full((B, len(heads), len(rows), K), -1, dtype=np.int64)
    gap = np.full((B, len(heads), len(rows)), POS_INF)
    for b in range(B):
        for hi, h in enumerate(heads):
            kh = np.asarray(k[b, h], dtype=np.float64)
            for ri, r in enumerate(rows):
                t = N - Nq + r
                res = selection_quality_row(q[b, h * G:(h + 1) * G, r], kh, block_idx[b, hi, ri], t, C, K, causal)
                met[b, hi, ri] = (res["recall"], res["captured"], res["ratio"])
                ref[b, hi, ri, :len(res["ref"])] = res["ref"]
                gap[b, hi, ri] = res["gap"]
    return met, ref, gap


def sparse_attention_bwd(q, k, v, block_idx, do, C, causal):
    """Gradients of the selected attention for every row and head (indices
    fixed): q, do [B, H, Nq, d]; k, v [B, Hkv, N, d]; block_idx [B, Hkv, Nq, K].
    Returns (dq [B, H, Nq, d], dk [B, Hkv, N, d], dv [B, Hkv, N, d]), float64;
    dk and dv sum the contributions of every query head of the KV group."""
    B, H, Nq, d = q.shape
    _, Hkv, N, _ = k.shape
    G = _group(H, Hkv)
    dq = np.zeros((B, H, Nq, d))
    dk = np.zeros((B, Hkv, N, d))
    dv = np.zeros((B, Hkv, N, d))
    for b in range(B):
        for hq in range(H):
            hk = hq // G
            kh = np.asarray(k[b, hk], dtype=np.float64)
            vh = np.asarray(v[b, hk], dtype=np.float64)
            for r in range(Nq):
                t = N - Nq + r
                g_q, tok, g_k, g_v = attention_row_bwd(q[b, hq, r], kh, vh, block_idx[b, hk, r], t, C, causal,
                                                       do[b, hq, r])
                dq[b, hq, r] = g_q
                if tok:
                    dk[b, hk, tok] += g_k
                    dv[b, hk, tok] += g_v
    return dq, dk, dv
