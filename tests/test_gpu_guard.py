"""Guard bands around every output and workspace, through the C ABI.

Each buffer an entry point writes (outputs and the caller's workspace) sits
in the middle of a larger allocation whose leading and trailing 4 KiB are
filled with a sentinel byte; after the call every sentinel byte must be
unchanged, and the results must equal those of the same call on ordinary
(unguarded) buffers.  An out-of-bounds write that does not fault shows up
here.  Covered: the pyramid build and decode append, every selection
schedule (with block scores), flat BSA, every attention path, the backward
and the selection-quality diagnostic, on parity shapes and on the
needles-128k workload at full size.
"""
import numpy as np
import pytest
import torch

from paper_2609_31093_amd import inputs
from tests.helpers import dev

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None

GUARD = 4096
SENT = 0xA5


class Guarded:
    """A device buffer of `nbytes` with sentinel-filled guard bands on both sides."""

    def __init__(self, nbytes, dtype=torch.uint8, shape=None):
        nbytes = int(nbytes)
        self.nbytes = nbytes
        pad = (-nbytes) % 256
        self.raw = torch.full((GUARD + nbytes + pad + GUARD,), SENT, dtype=torch.uint8, device="cuda")
        mid = self.raw[GUARD:GUARD + nbytes]
        self.t = mid.view(dtype).reshape(shape) if shape is not None else mid
        self.end = GUARD + nbytes

    def ptr(self):
        return self.t.data_ptr() if self.nbytes else None

    def check(self, what):
        torch.cuda.synchronize()
        lo = self.raw[:GUARD]
        hi = self.raw[self.end:]
        assert bool((lo == SENT).all()), f"{what}: write before the buffer"
        assert bool((hi == SENT).all()), f"{what}: write past the end of the buffer"


def _out(shape, dtype):
    n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    return Guarded(n, dtype, shape)


SHAPES = {
    # name: (B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    "gqa-ragged-bf16": (2, 8, 2, 2085, 2085, 128, 32, 2, 8, 1, "bf16"),
    "decode-row": (1, 4, 4, 1, 10000, 128, 64, 2, 8, 1, "bf16"),
    "tiny-fp32": (1, 2, 2, 1500, 1500, 64, 64, 2, 4, 1, "f32"),
    "k40-causal-block": (1, 4, 2, 5000, 5000, 64, 32, 2, 40, 1, "bf16"),
    "c128-g4-gqa": (1, 8, 2, 6000, 6000, 128, 128, 4, 8, 1, "bf16"),
    "noncausal-c128-ragged": (1, 4, 2, 900, 900, 64, 128, 2, 4, 0, "bf16"),
    "wide-g4-k32": (1, 4, 2, 9000, 9000, 128, 32, 4, 32, 1, "bf16"),
}


def _run_guarded(p, q, k, v, schedules, with_bwd, with_quality):
    B, H, Hkv, Nq, N, d, K = p.B, p.H, p.Hkv, p.Nq, p.N, p.d, p.K
    tdt = q.dtype
    # pyramid
    _, R = pisa.pisa_pyramid_layout(p)
    pyr = _out((B, Hkv, R, d), torch.float32)
    pisa.pisa_build_pyramid(p, k, pyr.ptr())
    pyr.check("pisa_build_pyramid")
    ref_pyr = pisa.build_pyramid(p, k)
    torch.cuda.synchronize()
    assert torch.equal(pyr.t, ref_pyr)
    # decode-cache append over the last 37 tokens (or all of them)
    n_old = max(0, N - 37)
    pyr2 = _out((B, Hkv, R, d), torch.float32)
    if n_old > 0:
        p_old = pisa.make_problem(B, H, Hkv, min(Nq, n_old), n_old, d, p.C, p.fanout, K, p.causal, tdt, Ncap=N)
        pisa.pisa_build_pyramid(p_old, k, pyr2.ptr())
    pisa.pisa_pyramid_append(p, k, pyr2.ptr(), n_old)
    pyr2.check("pisa_pyramid_append")
    assert torch.equal(pyr2.t, ref_pyr)
    # decode-cache growth into buffers for 1.5x the tokens (pyramid, k and v)
    new_cap = pisa.pisa_cache_capacity(N, N + 1, p.C)
    pn = pisa.make_problem(B, H, Hkv, Nq, N, d, p.C, p.fanout, K, p.causal, tdt, Ncap=new_cap)
    _, Rn = pisa.pisa_pyramid_layout(pn)
    gp = _out((B, Hkv, Rn, d), torch.float32)
    gk = _out((B, Hkv, new_cap, d), tdt)
    gv = _out((B, Hkv, new_cap, d), tdt)
    pisa.pisa_cache_grow(p, new_cap, pyr.ptr(), gp.ptr(), k, gk.ptr(), v, gv.ptr())
    for buf, what in ((gp, "pyramid"), (gk, "k"), (gv, "v")):
        buf.check(f"pisa_cache_grow {what}")
    assert torch.equal(gk.t[:, :, :N], k) and torch.equal(gv.t[:, :, :N], v)
    # selection, every requested schedule, with block scores
    idx_ref = None
    for sched in schedules:
        ps = pisa.make_problem(B, H, Hkv, Nq, N, d, p.C, p.fanout, K, p.causal, tdt, sched)
        nb = pisa.pisa_select_workspace_bytes(ps)
        ws = Guarded(nb)
        idx = _out((B, Hkv, Nq, K), torch.int32)
        sc = _out((B, Hkv, Nq, K), torch.float32)
        pisa.pisa_select(ps, q, k, pyr.ptr(), idx.ptr(), sc.ptr(), ws.ptr(), nb)
        for buf, what in ((idx, "block_idx"), (sc, "block_score"), (ws, "select workspace")):
            buf.check(f"pisa_select schedule {sched} {what}")
        want_idx, want_sc = pisa.select(ps, q, k, ref_pyr, with_score=True)
        torch.cuda.synchronize()
        assert torch.equal(idx.t, want_idx) and torch.equal(sc.t, want_sc), sched
        if sched == 0:
            idx_ref = want_idx
    # flat BSA
    nb = pisa.pisa_bsa_workspace_bytes(p)
    ws = Guarded(nb)
    bidx = _out((B, Hkv, Nq, K), torch.int32)
    pisa.pisa_select_flat_bsa(p, q, pyr.ptr(), bidx.ptr(), ws.ptr(), nb)
    bidx.check("pisa_select_flat_bsa block_idx")
    ws.check("pisa_select_flat_bsa workspace")
    assert torch.equal(bidx.t, pisa.select_flat_bsa(p, q, ref_pyr))
    # attention
    nb = pisa.pisa_attn_workspace_bytes(p)
    ws = Guarded(nb)
    o = _out(tuple(q.shape), tdt)
    lse = _out((B, H, Nq), torch.float32)
    pisa.pisa_sparse_attn_fwd(p, q, k, v, idx_ref, o.ptr(), lse.ptr(), ws.ptr(), nb)
    for buf, what in ((o, "o"), (lse, "lse"), (ws, "attention workspace")):
        buf.check(f"pisa_sparse_attn_fwd {what}")
    want_o, want_lse = pisa.sparse_attn_fwd(p, q, k, v, idx_ref)
    torch.cuda.synchronize()
    assert torch.equal(o.t, want_o) and torch.equal(lse.t, want_lse)
    if with_bwd:
        d_o = torch.randn(q.shape, generator=torch.Generator(device="cuda").manual_seed(3), device="cuda").to(tdt)
        nb = pisa.pisa_attn_bwd_workspace_bytes(p)
        ws = Guarded(nb)
        dq, dk, dv = _out(tuple(q.shape), tdt), _out(tuple(k.shape), tdt), _out(tuple(v.shape), tdt)
        pisa.pisa_sparse_attn_bwd(p, q, k, v, idx_ref, want_o, want_lse, d_o, dq.ptr(), dk.ptr(), dv.ptr(), ws.ptr(),
                                  nb)
        for buf, what in ((dq, "dq"), (dk, "dk"), (dv, "dv"), (ws, "backward workspace")):
            buf.check(f"pisa_sparse_attn_bwd {what}")
        wq, wk, wv = pisa.sparse_attn_bwd(p, q, k, v, idx_ref, want_o, want_lse, d_o)
        torch.cuda.synchronize()
        # the backward adds fp32 partials with atomics: equal up to summation order
        for got, want in ((dq, wq), (dk, wk), (dv, wv)):
            assert torch.allclose(got.t.float(), want.float(), rtol=2e-2, atol=2e-2 * float(want.float().abs().max()))
    if with_quality:
        rows = torch.tensor([0, Nq // 3, Nq - 1], dtype=torch.int32, device="cuda")
        nb = pisa.pisa_quality_workspace_bytes(p, 3)
        ws = Guarded(nb)
        met = _out((B, Hkv, 3, 3), torch.float32)
        ref = _out((B, Hkv, 3, K), torch.int32)
        pisa.pisa_selection_quality(p, q, k, idx_ref, rows, 3, met.ptr(), ref.ptr(), ws.ptr(), nb)
        for buf, what in ((met, "metrics"), (ref, "ref_idx"), (ws, "quality workspace")):
            buf.check(f"pisa_selection_quality {what}")
        wm, wr = pisa.selection_quality(p, q, k, idx_ref, rows)
        torch.cuda.synchronize()
        assert torch.equal(met.t, wm) and torch.equal(ref.t, wr)


@pytest.mark.parametrize("name", list(SHAPES))
def test_guard_bands(name):
    B, H, Hkv, Nq, N, d, C, g, K, causal, dtype = SHAPES[name]
    print("shape", SHAPES[name], flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, dtype, seed=17)
    q, k, v = dev(x["q"], dtype), dev(x["k"], dtype), dev(x["v"], dtype)
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, causal, dtype)
    schedules = (0, 1, 2, 3) if dtype == "bf16" else (0, 2, 3)
    bwd = dtype == "bf16" and C in (32, 64, 96, 128)
    qual = dtype == "bf16" and C in (32, 64, 96, 128) and K <= 64
    _run_guarded(p, q, k, v, schedules, bwd, qual)


def test_guard_bands_fullsize_needles():
    """The bench workload (needles-128k) in the bench's launch configuration."""
    w = inputs.workload("needles-128k")
    x = inputs.make_inputs(w, seed=0)
    q, k, v = (torch.from_numpy(x[n]).to(torch.bfloat16).cuda() for n in "qkv")
    p = pisa.make_problem(w["B"], w["H"], w["Hkv"], w["Nq"], w["N"], w["d"], w["C"], w["g"], w["K"], 1, "bf16")
    _run_guarded(p, q, k, v, (0,), with_bwd=False, with_quality=False)
