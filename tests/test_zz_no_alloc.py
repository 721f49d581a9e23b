"""pisa_select_static (the selection without a caller workspace, for callers
that cannot allocate) against pisa_select, through the C ABI.

Two calls in a row on shapes that use the static scratch (two-stage prefill,
then a smaller one; a decode step on the split schedule, then a smaller one),
each compared with pisa_select on the same inputs: indices and block scores
bit for bit (the same kernels on the same data).  A problem needing more
scratch than the array holds is refused with PISA_ERR_WORKSPACE and leaves
its outputs untouched.
"""
import numpy as np
import pytest
import torch

from paper_2609_31093_amd import inputs

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None


def _case(shape, seed, schedule=0):
    B, H, Hkv, Nq, N, d, C, g, K = shape
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=seed)
    q, k = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qk")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16", schedule)
    return p, q, k, pisa.build_pyramid(p, k)


def _static(p, q, k, pyr):
    idx = torch.full((p.B, p.Hkv, p.Nq, p.K), -7, dtype=torch.int32, device="cuda")
    sc = torch.full((p.B, p.Hkv, p.Nq, p.K), 7.0, dtype=torch.float32, device="cuda")
    pisa.pisa_select_static(p, q, k, pyr, idx, sc)
    return idx, sc


PAIRS = {
    # first call, then a smaller second call (both within the static scratch)
    "two-stage": ((1, 8, 4, 8192, 8192, 128, 64, 2, 16), (1, 4, 2, 3000, 5000, 64, 32, 2, 8)),
    "split-decode": ((1, 8, 8, 1, 131072, 128, 64, 2, 16), (1, 4, 2, 1, 7000, 128, 64, 2, 6)),
    "wide-two-stage": ((1, 8, 2, 6000, 6000, 128, 32, 4, 16), (1, 2, 1, 4096, 4096, 64, 64, 2, 24)),
}


@pytest.mark.parametrize("name", list(PAIRS))
def test_select_static_matches_select(name):
    for i, shape in enumerate(PAIRS[name]):
        p, q, k, pyr = _case(shape, seed=40 + i)
        need = pisa.pisa_select_workspace_bytes(p)
        assert 0 < need <= pisa.PISA_STATIC_SCRATCH_BYTES, (shape, need)
        got_idx, got_sc = _static(p, q, k, pyr)
        want_idx, want_sc = pisa.select(p, q, k, pyr, with_score=True)
        torch.cuda.synchronize()
        assert torch.equal(got_idx, want_idx), (name, i)
        assert torch.equal(got_sc, want_sc), (name, i)


def test_select_static_refuses_beyond_the_scratch():
    shape = (1, 8, 8, 32768, 32768, 128, 64, 2, 16)
    p, q, k, pyr = _case(shape, seed=50)
    assert pisa.pisa_select_workspace_bytes(p) > pisa.PISA_STATIC_SCRATCH_BYTES
    idx = torch.full((p.B, p.Hkv, p.Nq, p.K), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(pisa.PisaError) as e:
        pisa.pisa_select_static(p, q, k, pyr, idx, None)
    assert e.value.status == pisa.PISA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((idx == -7).all())
    # and a fitting call afterwards still matches pisa_select
    p2, q2, k2, pyr2 = _case((1, 4, 4, 4096, 4096, 128, 64, 2, 16), seed=51)
    got, _ = _static(p2, q2, k2, pyr2)
    torch.cuda.synchronize()
    assert torch.equal(got, pisa.select(p2, q2, k2, pyr2))
