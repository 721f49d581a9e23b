"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Acceptance:
  * pyramid: |gpu - oracle| <= the per-node float32 bound of
    tests/helpers.py pyramid_error_bound on every element (mean of means)
  * indices: identical on every sampled row whose oracle margin exceeds 1e-3;
    on the other sampled rows identical or an admissible selection (the
    oracle's near-tie replay, exact ties to the smaller index), and every row
    of every output a valid selection
  * block_score: the oracle's grouped raw-key score of each scored kept block
    within 1e-3, +inf for blocks kept without a score, -inf at padding
  * attention on the GPU's own indices: o within 2e-2 (bf16) / 1e-4 (fp32)
    max-abs, lse within 1e-3.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import (check_flat_bsa_rows, check_selection_rows, check_selection_valid, check_valid_all_rows, dev,
                           pyramid_error_bound)

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:  # collected on CPU only to be deselected by -m "not gpu"
    pisa = None


def _rows_sample(Nq, n_edge=48, n_mid=64, seed=0):
    if Nq <= 2 * n_edge + n_mid:
        return np.arange(Nq)
    r = np.random.default_rng(seed)
    mid = r.choice(np.arange(n_edge, Nq - n_edge), size=n_mid, replace=False)
    return np.unique(np.concatenate([np.arange(n_edge), mid, np.arange(Nq - n_edge, Nq)]))


SHAPES = {
    # name: (B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    "tiny-fp32": (1, 2, 2, 4096, 4096, 64, 64, 2, 4, 1, "f32"),
    "gqa-ragged-bf16": (2, 8, 2, 2085, 2085, 128, 32, 2, 8, 1, "bf16"),
    "g4-gqa4-d64": (1, 4, 1, 5000, 5000, 64, 64, 4, 6, 1, "bf16"),
    "g3-noncausal": (1, 2, 2, 3000, 3000, 128, 32, 3, 5, 0, "bf16"),
    "suffix-rows": (1, 2, 1, 300, 4000, 128, 64, 2, 5, 1, "bf16"),
    "single-block": (1, 2, 2, 50, 50, 64, 64, 2, 3, 1, "f32"),
    "decode-row": (1, 4, 4, 1, 10000, 128, 64, 2, 8, 1, "bf16"),
    "big-budget": (1, 2, 2, 2048, 2048, 64, 32, 2, 64, 1, "f32"),
    "noncausal-f32-ragged": (1, 2, 1, 777, 777, 64, 32, 2, 4, 0, "f32"),
    "c128-g4-gqa": (1, 8, 2, 6000, 6000, 128, 128, 4, 8, 1, "bf16"),
    # bf16 row counts between the split and the block-centric attention paths
    "mid-rows-bf16": (1, 4, 2, 1500, 1500, 64, 32, 2, 6, 1, "bf16"),
    # few rows (split paths) with GQA, C = 128 and no causal mask
    "split-gqa-c128-noncausal": (1, 8, 2, 700, 5000, 128, 128, 2, 6, 0, "bf16"),
    # no causal mask, so the 4-key last block is scored: key tiles with no key
    "noncausal-c128-ragged": (1, 4, 2, 900, 900, 64, 128, 2, 4, 0, "bf16"),
    # fan-out 2 stage 1 with one head per KV head at d = 64, and with three heads per group
    "mha-d64-bf16": (1, 2, 2, 3000, 3000, 64, 32, 2, 8, 1, "bf16"),
    "gqa3-bf16": (1, 6, 2, 2500, 2500, 128, 64, 2, 8, 1, "bf16"),
    # g*K > 32: stage 1 on the matrix cores (fan-out 4 and 2, one to four heads per KV head)
    "wide-g4-gqa4": (1, 8, 2, 4000, 4000, 128, 32, 4, 12, 1, "bf16"),
    "wide-g2-d64": (1, 2, 2, 5000, 5000, 64, 32, 2, 24, 1, "bf16"),
    "wide-g4-k32": (1, 4, 2, 9000, 9000, 128, 32, 4, 32, 1, "bf16"),
    "wide-g4-noncausal-suffix": (1, 4, 1, 1500, 3000, 128, 32, 4, 10, 0, "bf16"),
    # sixteen and eight query heads per KV head (the paper's benchmark grouping)
    "gqa16-d64-k8": (1, 32, 2, 3000, 3000, 64, 64, 2, 8, 1, "bf16"),
    "gqa8-g4-c32": (1, 16, 2, 4000, 4000, 128, 32, 4, 6, 1, "bf16"),
    # causal budgets above 32 on the block attention path (slots 32.. merged after the per-leaf-block kernel)
    "k40-causal-block": (1, 4, 2, 5000, 5000, 64, 32, 2, 40, 1, "bf16"),
    "k48-causal-block-d128": (1, 2, 1, 6000, 6000, 128, 64, 2, 48, 1, "bf16"),
    # leaf blocks above 128 keys (query-centric attention; the general leaf scorer with > 64 KiB of LDS)
    "c256-two-stage": (1, 4, 2, 3000, 6000, 128, 256, 2, 6, 1, "bf16"),
    "c160-g3-noncausal": (1, 2, 1, 2500, 2500, 64, 160, 3, 5, 0, "bf16"),
}


def _problem(shape, schedule=0, score=0):
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    return pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype, schedule, score=score)


def _data(shape, seed=0):
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    return inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=seed)


@pytest.mark.parametrize("name", list(SHAPES))
def test_pyramid_parity(name):
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    x = _data(shape)
    p = _problem(shape)
    pyr = pisa.build_pyramid(p, dev(x["k"], dtype))
    torch.cuda.synchronize()
    want = O.pyramid(x["k"], C, g)
    err = np.abs(pyr.cpu().numpy() - want)
    bound = pyramid_error_bound(x["k"], C, g)
    print("pyramid max err / bound", float((err / bound).max()), flush=True)
    assert np.all(err <= bound), float((err - bound).max())


# Long sequences whose top pyramid levels do (g = 4, 4096 leaves: 160 KiB) or
# do not (g = 2, 4096 leaves: 192 KiB) fit the LDS of the top-level pooling
# workgroup, so that both of its variants are compared with the oracle.
LARGE_PYRAMIDS = {
    "top-levels-in-lds-g4": (1, 1, 1, 16, 524288, 128, 128, 4, 8, 1, "bf16"),
    "top-levels-global-g2": (1, 1, 1, 16, 262144, 128, 64, 2, 8, 1, "bf16"),
}


@pytest.mark.parametrize("name", list(LARGE_PYRAMIDS))
def test_pyramid_parity_large(name):
    shape = LARGE_PYRAMIDS[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    x = _data(shape)
    p = _problem(shape)
    pyr = pisa.build_pyramid(p, dev(x["k"], dtype))
    torch.cuda.synchronize()
    want = O.pyramid(x["k"], C, g)
    err = np.abs(pyr.cpu().numpy() - want)
    bound = pyramid_error_bound(x["k"], C, g)
    print("pyramid max err / bound", float((err / bound).max()), flush=True)
    assert np.all(err <= bound), float((err - bound).max())


def _run_select(shape, schedule, x, score=0):
    p = _problem(shape, schedule, score)
    dtype = shape[-1]
    q, k = dev(x["q"], dtype), dev(x["k"], dtype)
    pyr = pisa.build_pyramid(p, k)
    idx, sc = pisa.select(p, q, k, pyr, with_score=True)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), sc.cpu().numpy()


SCHEDULES = (2, 1, 3)  # fused, two-stage, split


@pytest.mark.parametrize("name", list(SHAPES))
@pytest.mark.parametrize("schedule", SCHEDULES, ids=["fused", "two_stage", "split"])
def test_select_parity(name, schedule):
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    if schedule == 1 and dtype != "bf16":
        pytest.skip("two-stage schedule is bf16-only")
    x = _data(shape)
    idx, sc = _run_select(shape, schedule, x)
    check_selection_valid(idx, N, Nq, C, K, bool(causal))
    rows = _rows_sample(Nq)
    stats = check_selection_rows(x["q"], x["k"], C, g, K, bool(causal), idx[:, :, rows], rows,
                                 gpu_score=sc[:, :, rows])
    print(name, schedule, stats)
    # every row: -inf exactly at padding
    assert np.all(np.isneginf(sc) == (idx < 0))


def test_schedules_agree_on_decisive_rows():
    shape = SHAPES["gqa-ragged-bf16"]
    x = _data(shape, seed=3)
    a, _ = _run_select(shape, 2, x)
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    rows = _rows_sample(Nq, 16, 32)
    _, gap = O.select(x["q"], x["k"], C, g, K, bool(causal), rows=rows)
    for other in (1, 3):
        b, _ = _run_select(shape, other, x)
        assert not ((a[:, :, rows] != b[:, :, rows]).any(-1) & (gap > 1e-3)).any(), other


@pytest.mark.parametrize("name", list(SHAPES))
def test_attention_parity_on_gpu_indices(name):
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    x = _data(shape)
    p = _problem(shape)
    q, k, v = dev(x["q"], dtype), dev(x["k"], dtype), dev(x["v"], dtype)
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    rows = _rows_sample(Nq, 32, 48)
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, bool(causal), rows=rows)
    got_o = o.float().cpu().numpy()[:, :, rows]
    got_lse = lse.cpu().numpy()[:, :, rows]
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.abs(got_o - want_o).max() <= tol
    assert np.abs(got_lse - want_lse).max() <= 1e-3


@pytest.mark.parametrize("causal", [1, 0])
def test_attention_all_blocks_is_dense(causal):
    """K*C >= N: selected attention equals dense (causal) softmax attention."""
    B, H, Hkv, N, d, C = 1, 4, 2, 700, 64, 32
    M1 = -(-N // C)
    shape = (B, H, Hkv, N, N, d, C, 2, M1, causal, "f32")
    x = _data(shape, seed=5)
    p = _problem(shape)
    idx = torch.arange(M1, dtype=torch.int32).repeat(B, Hkv, N, 1).contiguous().cuda()
    o, lse = pisa.sparse_attn_fwd(p, dev(x["q"], "f32"), dev(x["k"], "f32"), dev(x["v"], "f32"), idx)
    torch.cuda.synchronize()
    G = H // Hkv
    qd = torch.from_numpy(x["q"]).double()
    kd = torch.from_numpy(x["k"]).double().repeat_interleave(G, dim=1)
    vd = torch.from_numpy(x["v"]).double().repeat_interleave(G, dim=1)
    want = torch.nn.functional.scaled_dot_product_attention(qd, kd, vd, is_causal=bool(causal))
    z = qd @ kd.transpose(-1, -2) / math.sqrt(d)
    if causal:
        z = z.masked_fill(~torch.ones(N, N, dtype=torch.bool).tril(), -math.inf)
    assert (o.double().cpu() - want).abs().max().item() <= 1e-4
    assert (lse.double().cpu() - torch.logsumexp(z, -1)).abs().max().item() <= 1e-3


@pytest.mark.parametrize("name", ["tiny-fp32", "gqa-ragged-bf16", "g4-gqa4-d64", "g3-noncausal", "suffix-rows"])
def test_flat_bsa_parity(name):
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    x = _data(shape, seed=7)
    p = _problem(shape)
    q, k = dev(x["q"], dtype), dev(x["k"], dtype)
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select_flat_bsa(p, q, pyr)
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    check_selection_valid(idx, N, Nq, C, K, bool(causal))
    rows = _rows_sample(Nq)
    print(name, check_flat_bsa_rows(x["q"], x["k"], C, K, bool(causal), idx[:, :, rows], rows))


def test_deterministic_repeat():
    shape = SHAPES["gqa-ragged-bf16"]
    x = _data(shape, seed=11)
    p = _problem(shape)
    q, k, v = (dev(x[n], "bf16") for n in "qkv")
    outs = []
    for _ in range(2):
        pyr = pisa.build_pyramid(p, k)
        idx = pisa.select(p, q, k, pyr)
        o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
        bsa = pisa.select_flat_bsa(p, q, pyr)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (pyr, idx, o, lse, bsa)])
    for a, b in zip(*outs):
        assert torch.equal(a, b)


VARIANT_SHAPES = ["tiny-fp32", "gqa-ragged-bf16", "g4-gqa4-d64", "decode-row", "c128-g4-gqa", "big-budget",
                  "noncausal-c128-ragged", "g3-noncausal", "wide-g4-gqa4", "wide-g2-d64", "gqa16-d64-k8"]


@pytest.mark.parametrize("name", VARIANT_SHAPES)
@pytest.mark.parametrize("score", [1, 2], ids=["pisa1-mean", "pisa2-mean-var"])
@pytest.mark.parametrize("schedule", SCHEDULES, ids=["fused", "two_stage", "split"])
def test_select_parity_score_variants(name, score, schedule):
    """PISA-1 / PISA-2 (App. A) through every schedule, against the oracle."""
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    if schedule == 1 and dtype != "bf16":
        pytest.skip("two-stage schedule is bf16-only")
    x = _data(shape, seed=7)
    idx, sc = _run_select(shape, schedule, x, score)
    check_selection_valid(idx, N, Nq, C, K, bool(causal))
    rows = _rows_sample(Nq, 24, 32)
    stats = check_selection_rows(x["q"], x["k"], C, g, K, bool(causal), idx[:, :, rows], rows,
                                 gpu_score=sc[:, :, rows], score={1: "mean", 2: "mean_var"}[score])
    print(name, score, schedule, stats)
    assert np.all(np.isneginf(sc) == (idx < 0))
    assert np.all(np.isfinite(sc) | np.isinf(sc))



def _plant_out_of_range(idx_np, N, Nq, C, causal):
    """Overwrite the last slot of every row with an entry that must contribute
    nothing: a block past the end (M1 + small, or ~2^30), or (causal) a block
    that starts after the query."""
    M1 = -(-N // C)
    out = idx_np.copy()
    for r in range(Nq):
        t = N - Nq + r
        c = t // C
        kind = r % 3
        if kind == 0:
            val = M1 + (r % 7)
        elif kind == 1:
            val = (1 << 30) - r
        else:
            val = min(c + 1 + r % 5, M1 - 1) if causal and c + 1 < M1 else -1
        out[..., r, -1] = val
    return out


@pytest.mark.parametrize("name", ["gqa-ragged-bf16", "k40-causal-block", "decode-row", "tiny-fp32",
                                  "split-gqa-c128-noncausal"])
def test_attention_out_of_range_indices_are_padding(name):
    """Entries at or past ceil(N/C) (and, causal, blocks after the query) add
    nothing on every attention path (block-centric, split, query-centric)."""
    shape = SHAPES[name]
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = shape
    x = _data(shape, seed=13)
    p = _problem(shape)
    q, k, v = dev(x["q"], dtype), dev(x["k"], dtype), dev(x["v"], dtype)
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    torch.cuda.synchronize()
    planted = _plant_out_of_range(idx.cpu().numpy(), N, Nq, C, bool(causal))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, torch.from_numpy(planted).cuda())
    torch.cuda.synchronize()
    rows = _rows_sample(Nq, 16, 32)
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], planted[:, :, rows], C, bool(causal), rows=rows)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert np.abs(o.float().cpu().numpy()[:, :, rows] - want_o).max() <= tol
    assert np.abs(lse.cpu().numpy()[:, :, rows] - want_lse).max() <= 1e-3


@pytest.mark.parametrize("G", [1, 4])
def test_flat_bsa_all_scores_tied(G):
    """Every key equal: every block scores the same, so each row keeps its
    forced blocks plus the smallest eligible ones (reading R4).  More tied
    blocks rank at the cut than the fast threshold method collects, so its
    exact fallback runs (single head, more than 8 chunks of 64 blocks)."""
    B, Hkv, Nq, N, d, C, K = 1, 2, 600, 40000, 64, 32, 16
    H = G * Hkv
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=21)
    x["k"][:] = x["k"][:, :, :1, :]
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, 1, "bf16")
    q, k = dev(x["q"], "bf16"), dev(x["k"], "bf16")
    idx = pisa.select_flat_bsa(p, q, pisa.build_pyramid(p, k))
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    check_selection_valid(idx, N, Nq, C, K, True)
    rows = _rows_sample(Nq, 8, 16)
    print(check_flat_bsa_rows(x["q"], x["k"], C, K, True, idx[:, :, rows], rows))
    for r in rows:
        c = (N - Nq + r) // C
        want = sorted({0, c - 1, c} | set(range(1, K - 2)))   # K - 3 unforced: blocks 1 .. K - 3
        assert list(idx[0, 0, r]) == want, (r, idx[0, 0, r])


def test_select_large_ragged_grid():
    """A grid past 65536 (batch x KV head x row) rows whose count is not a
    multiple of the final Top-K's rows per workgroup (16 there, two row pairs
    per wavefront): the last rows and sampled others against the oracle, and
    every row a valid selection."""
    B, H, Hkv, N, d, C, g, K = 1, 1, 1, 65541, 128, 64, 2, 16
    x = inputs.random_qkv(B, H, Hkv, N, N, d, "bf16", seed=21)
    q, k = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qk")
    p = pisa.make_problem(B, H, Hkv, N, N, d, C, g, K, 1, "bf16")
    assert (B * Hkv * N) % 16 != 0 and B * Hkv * N >= 65536
    idx, sc = pisa.select(p, q, k, pisa.build_pyramid(p, k), with_score=True)
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    check_valid_all_rows(idx_np, N, N, C, K, True)
    rows = np.unique(np.concatenate([np.arange(N - 18, N), np.random.default_rng(22).choice(N, 14, replace=False)]))
    check_selection_rows(x["q"], x["k"], C, g, K, True, idx_np[:, :, rows], rows, gpu_score=sc.cpu().numpy()[:, :, rows])
