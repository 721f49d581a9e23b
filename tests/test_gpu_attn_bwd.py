"""GPU parity of the sparse-attention backward with the selection held fixed
(App. B) against the oracle's gradients (float64, written from the gradient
definitions and pinned to torch autograd), through the C ABI.

The backward gets the GPU's own selection and forward outputs (o, lse); the
oracle gets the same selection.  Tolerance (bf16 inputs and outputs): every
gradient within 2% of that tensor's largest oracle magnitude.  Derivation:
the kernels round P and dS to bf16 for the matrix-core products (relative
2^-9 each), keep each (row, block) dq term in bf16 before the sum (2^-9), sum
in fp32 and round the result to bf16 (2^-9); with 16-64 terms of mixed sign
the worst element stays well inside 2% of the tensor's scale.
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

REL = 2e-2

SHAPES = {
    # name: (B, H, Hkv, Nq, N, d, C, K, causal)
    "gqa2-c64": (1, 4, 2, 1200, 1200, 128, 64, 6, 1),
    "mha-c32-d64": (2, 2, 2, 700, 700, 64, 32, 5, 1),
    "gqa4-c128-d64": (1, 8, 2, 1000, 1000, 64, 128, 4, 1),
    "noncausal-c96": (1, 2, 1, 700, 800, 128, 96, 5, 0),
    "c128-d128": (1, 2, 2, 1100, 1100, 128, 128, 4, 1),  # dq operand read from row-major K
    "suffix-rows": (1, 2, 1, 300, 3000, 128, 64, 8, 1),
}


def _grads(shape, seed):
    B, H, Hkv, Nq, N, d, C, K, causal = shape
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=seed)
    do_np = inputs.round_to_bf16(np.random.default_rng(seed + 100).standard_normal((B, H, Nq, d)).astype(np.float32))
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    d_o = torch.from_numpy(do_np).to(torch.bfloat16).cuda()
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, causal, "bf16")
    pyr = pisa.build_pyramid(p, k)
    idx = pisa.select(p, q, k, pyr)
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    torch.cuda.synchronize()
    want = O.sparse_attention_bwd(x["q"], x["k"], x["v"], idx.cpu().numpy(), do_np, C, bool(causal))
    got = [t.float().cpu().numpy() for t in (dq, dk, dv)]
    return got, want


@pytest.mark.parametrize("name", list(SHAPES))
def test_attention_backward_parity(name):
    got, want = _grads(SHAPES[name], seed=5)
    for label, g, w in zip(("dq", "dk", "dv"), got, want):
        scale = float(np.abs(w).max())
        err = float(np.abs(g - w).max())
        assert scale > 0, label
        assert err <= REL * scale, (label, err, scale)
        print(f"{name} {label}: max|err| {err:.3e} of scale {scale:.3e}")


def test_attention_backward_untouched_rows_are_zero():
    """Keys no query selects (the suffix rows only reach their own recent blocks
    and the forced ones) get exactly zero gradient."""
    B, H, Hkv, Nq, N, d, C, K = 1, 2, 1, 64, 4096, 128, 64, 3
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=6)
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    d_o = torch.randn((B, H, Nq, d), device="cuda").to(torch.bfloat16)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, 1, "bf16")
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    torch.cuda.synchronize()
    reached = torch.zeros(N, dtype=torch.bool)
    for blk in idx.cpu().unique().tolist():
        if blk >= 0:
            reached[blk * C:(blk + 1) * C] = True
    assert (dk[0, 0, ~reached.cuda()] == 0).all() and (dv[0, 0, ~reached.cuda()] == 0).all()
    assert (dk[0, 0, reached.cuda()] != 0).any()


def test_attention_backward_reserved_rows():
    """With rows reserved past N (Ncap > N, the decode cache's layout; the
    reserved k and v rows hold NaN), dq equals the unreserved run's bit for
    bit, dk and dv on rows [0, N) equal it up to the fp32 summation order (the
    pair order inside a block's cluster varies between runs), and dk, dv are
    zero on rows [N, Ncap) whatever the buffers held before."""
    B, H, Hkv, Nq, N, d, C, K, cap = 1, 4, 2, 700, 1000, 128, 64, 5, 1300
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=8)
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    d_o = torch.randn((B, H, Nq, d), device="cuda").to(torch.bfloat16)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, 1, "bf16")
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq0, dk0, dv0 = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    pc = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, 1, "bf16", Ncap=cap)
    kc = torch.full((B, Hkv, cap, d), float("nan"), device="cuda", dtype=torch.bfloat16)
    vc = kc.clone()
    kc[:, :, :N] = k
    vc[:, :, :N] = v
    dq = torch.full_like(q, float("nan"))
    dk = torch.full_like(kc, float("nan"))
    dv = torch.full_like(vc, float("nan"))
    nb = pisa.pisa_attn_bwd_workspace_bytes(pc)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda")
    pisa.pisa_sparse_attn_bwd(pc, q, kc, vc, idx, o, lse, d_o, dq, dk, dv, ws, nb, None)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq0)
    for got, want in ((dk[:, :, :N], dk0), (dv[:, :, :N], dv0)):
        assert torch.allclose(got.float(), want.float(), rtol=2e-2, atol=2e-2 * float(want.float().abs().max()))
    assert (dk[:, :, N:] == 0).all() and (dv[:, :, N:] == 0).all()


def test_attention_backward_needles_128k():
    """At the needle workload's full size, in the launch configuration bench.py
    --backward times: dq of sampled rows against the oracle (a row's dq depends
    only on that row), and two identities that hold at any size, per KV head:
    sum_j dv_j = sum over rows and group heads of do (each row's p sums to
    one), and sum_j dk_j = 0 (each row's ds sums to zero)."""
    w = inputs.workload("needles-128k")
    x = inputs.make_inputs(w, seed=0)
    B, H, Hkv, N, Nq, d, C, g, K = (w[kk] for kk in ("B", "H", "Hkv", "N", "Nq", "d", "C", "g", "K"))
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    gen = torch.Generator(device="cuda").manual_seed(7)
    d_o = torch.randn((B, H, Nq, d), device="cuda", generator=gen).to(torch.bfloat16)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16")
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    torch.cuda.synchronize()
    # identities (fp64 sums of the bf16 gradients)
    sdv = dv.double().sum(2)
    sdo = d_o.double().view(B, Hkv, H // Hkv, Nq, d).sum((2, 3))
    assert (sdv - sdo).abs().max().item() <= 1e-2 * sdo.abs().max().item() + 1.0
    sdk = dk.double().sum(2)
    assert sdk.abs().max().item() <= 2e-3 * dk.double().abs().sum(2).max().item()
    # sampled rows against the oracle
    rows = [0, 1, 63, 64, 4097, Nq // 2, Nq - 1] + inputs.needle_layout(w)["qpos"][:3].tolist()
    do_np = d_o.float().cpu().numpy()
    sel = idx.cpu().numpy()
    want, got = [], []
    for h in (0, 5):
        kh, vh = x["k"][0, h].astype(np.float64), x["v"][0, h].astype(np.float64)
        for r in rows:
            t = N - Nq + r
            want.append(O.attention_row_bwd(x["q"][0, h, r], kh, vh, sel[0, h, r], t, C, True, do_np[0, h, r])[0])
            got.append(dq[0, h, r].float().cpu().numpy())
    want, got = np.array(want), np.array(got)
    # the same bound as the other shapes: 2% of the sampled rows' largest magnitude
    assert np.abs(got - want).max() <= REL * np.abs(want).max()


def test_attention_backward_across_row_chunks():
    """More (row, slot) pairs than one launch's partial budget (4 GiB of dq
    partials), so the rows go in four chunks and every key block adds into the
    fp32 accumulators across launches: sampled rows' dq against the oracle and
    the two per-KV-head identities of the full-size test."""
    B, H, Hkv, Nq, N, d, C, g, K = 1, 16, 2, 60000, 60000, 128, 64, 2, 64
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=12)
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    gen = torch.Generator(device="cuda").manual_seed(13)
    d_o = torch.randn((B, H, Nq, d), device="cuda", generator=gen).to(torch.bfloat16)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16")
    per_row = B * Hkv * K * (H // Hkv) * d * 2  # bytes of dq partials per row
    assert per_row * Nq > 3 * (4 << 30), "the shape must span several row chunks"
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, idx, o, lse, d_o)
    torch.cuda.synchronize()
    sdv = dv.double().sum(2)
    sdo = d_o.double().view(B, Hkv, H // Hkv, Nq, d).sum((2, 3))
    assert (sdv - sdo).abs().max().item() <= 1e-2 * sdo.abs().max().item() + 1.0
    sdk = dk.double().sum(2)
    assert sdk.abs().max().item() <= 2e-3 * dk.double().abs().sum(2).max().item()
    rows = [0, 1, 16383, 16384, 30000, 32768, Nq - 1]  # both sides of the chunk boundaries
    do_np = d_o.float().cpu().numpy()
    sel = idx.cpu().numpy()
    want, got = [], []
    for hq in (0, 11):
        hk = hq // (H // Hkv)
        kh, vh = x["k"][0, hk].astype(np.float64), x["v"][0, hk].astype(np.float64)
        for r in rows:
            t = N - Nq + r
            want.append(O.attention_row_bwd(x["q"][0, hq, r], kh, vh, sel[0, hk, r], t, C, True, do_np[0, hq, r])[0])
            got.append(dq[0, hq, r].float().cpu().numpy())
    want, got = np.array(want), np.array(got)
    assert np.abs(got - want).max() <= REL * np.abs(want).max()


def test_backward_out_of_range_indices_are_padding():
    """Entries at or past ceil(N/C) add nothing to any gradient."""
    B, H, Hkv, Nq, N, d, C, K, causal = SHAPES["gqa2-c64"]
    seed = 9
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=seed)
    do_np = inputs.round_to_bf16(np.random.default_rng(seed + 100).standard_normal((B, H, Nq, d)).astype(np.float32))
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    d_o = torch.from_numpy(do_np).to(torch.bfloat16).cuda()
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, causal, "bf16")
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    torch.cuda.synchronize()
    M1 = -(-N // C)
    planted = idx.cpu().numpy()
    planted[..., ::2, -1] = M1 + 3
    planted[..., 1::2, -1] = (1 << 30) - 1
    pidx = torch.from_numpy(planted).cuda()
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, pidx)
    dq, dk, dv = pisa.sparse_attn_bwd(p, q, k, v, pidx, o, lse, d_o)
    torch.cuda.synchronize()
    want = O.sparse_attention_bwd(x["q"], x["k"], x["v"], planted, do_np, C, bool(causal))
    for label, g, w in zip(("dq", "dk", "dv"), (dq, dk, dv), want):
        scale = float(np.abs(w).max())
        err = float(np.abs(g.float().cpu().numpy() - w).max())
        assert err <= REL * scale, (label, err, scale)
