"""C-ABI contract tests that need no GPU: the library loads, exports every
symbol the header declares, computes the hierarchy geometry, and rejects bad
arguments (exact status, non-empty detail) before anything is launched."""
import ctypes
import math
import os
import re
import subprocess

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pisa.h")

pisa = pytest.importorskip("paper_2609_31093_amd.pisa", reason="libpisa.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pisa_[a-z_]+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for must in ("pisa_build_pyramid", "pisa_select", "pisa_sparse_attn_fwd", "pisa_select_flat_bsa"):
        assert must in names
    assert set(names) == set(pisa.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = pisa.library()
    out = subprocess.run(["nm", "-D", "--defined-only", lib._name], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (pisa_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


@pytest.mark.parametrize("N,C,g", [(4096, 64, 2), (131072, 64, 2), (524288, 128, 4), (1025, 64, 2),
                                   (700, 32, 3), (64, 64, 2), (1, 32, 5)])
def test_num_levels_and_layout_match_hierarchy(N, C, g):
    sizes = O.level_sizes(N, C, g)
    assert pisa.pisa_num_levels(N, C, g) == len(sizes)
    p = pisa.make_problem(1, 2, 1, min(N, 16), N, 64, C, g, 3)
    offs, R = pisa.pisa_pyramid_layout(p)
    stored = sizes[:-1] if len(sizes) > 1 else sizes
    assert R == sum(stored)
    assert offs[0] == 0
    for lv in range(1, len(stored)):
        assert offs[lv] == sum(stored[:lv])
    assert pisa.pisa_pyramid_bytes(p) == 1 * 1 * R * 64 * 4


def _good(**kw):
    base = dict(B=1, H=4, Hkv=2, Nq=256, N=1024, d=128, C=64, fanout=2, K=4, causal=1, dtype="bf16")
    base.update(kw)
    return pisa.make_problem(**base)


FAKE = 1 << 20  # an aligned, non-null address; never dereferenced because validation fails first


BAD = [
    (dict(H=3, Hkv=2), pisa.PISA_ERR_INVALID_ARG),
    (dict(Nq=2048), pisa.PISA_ERR_INVALID_ARG),
    (dict(Nq=0), pisa.PISA_ERR_INVALID_ARG),
    (dict(K=2), pisa.PISA_ERR_INVALID_ARG),
    (dict(fanout=1), pisa.PISA_ERR_INVALID_ARG),
    (dict(causal=2), pisa.PISA_ERR_INVALID_ARG),
    (dict(d=96), pisa.PISA_ERR_UNSUPPORTED),
    (dict(C=48), pisa.PISA_ERR_UNSUPPORTED),
    (dict(C=512), pisa.PISA_ERR_UNSUPPORTED),
    (dict(fanout=17), pisa.PISA_ERR_UNSUPPORTED),
    (dict(fanout=16, K=17), pisa.PISA_ERR_UNSUPPORTED),
    (dict(H=68, Hkv=2), pisa.PISA_ERR_UNSUPPORTED),
    (dict(schedule=4), pisa.PISA_ERR_INVALID_ARG),
    (dict(Ncap=1000), pisa.PISA_ERR_INVALID_ARG),
    (dict(schedule=-1), pisa.PISA_ERR_INVALID_ARG),
]


@pytest.mark.parametrize("kw,status", BAD)
def test_invalid_problems_are_rejected_before_launch(kw, status):
    p = _good(**kw)
    calls = [
        lambda: pisa.library().pisa_build_pyramid(ctypes.byref(p), FAKE, FAKE, None),
        lambda: pisa.library().pisa_select(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 40, None),
        lambda: pisa.library().pisa_select_flat_bsa(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 1 << 40, None),
        lambda: pisa.library().pisa_sparse_attn_fwd(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                                     1 << 40, None),
    ]
    for call in calls:
        assert call() == status
        assert pisa.pisa_last_error() != ""
    assert pisa.pisa_pyramid_bytes(p) == 0
    assert pisa.pisa_select_workspace_bytes(p) == 0


def test_null_and_misaligned_pointers_are_rejected():
    p = _good()
    lib = pisa.library()
    assert lib.pisa_build_pyramid(ctypes.byref(p), None, FAKE, None) == pisa.PISA_ERR_INVALID_ARG
    assert "k" in pisa.pisa_last_error()
    assert lib.pisa_build_pyramid(ctypes.byref(p), FAKE + 2, FAKE, None) == pisa.PISA_ERR_INVALID_ARG
    assert "aligned" in pisa.pisa_last_error()
    assert lib.pisa_sparse_attn_fwd(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, None, None, 0, None) \
        == pisa.PISA_ERR_INVALID_ARG
    assert lib.pisa_select(None, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == pisa.PISA_ERR_INVALID_ARG


@pytest.mark.parametrize("schedule", [pisa.PISA_SCHEDULE_TWO_STAGE, pisa.PISA_SCHEDULE_SPLIT],
                         ids=["two_stage", "split"])
def test_undersized_workspace_is_rejected(schedule):
    p = _good(schedule=schedule)
    need = pisa.pisa_select_workspace_bytes(p)
    assert need > 0
    lib = pisa.library()
    st = lib.pisa_select(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, FAKE, need - 1, None)
    assert st == pisa.PISA_ERR_WORKSPACE
    assert str(need) in pisa.pisa_last_error()
    st = lib.pisa_select(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, None, need, None)
    assert st == pisa.PISA_ERR_WORKSPACE


def test_two_stage_needs_bf16():
    p = _good(dtype="f32", schedule=pisa.PISA_SCHEDULE_TWO_STAGE)
    lib = pisa.library()
    st = lib.pisa_select(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 40, None)
    assert st == pisa.PISA_ERR_UNSUPPORTED


def test_status_strings():
    assert pisa.pisa_status_string(0) == "ok"
    assert pisa.pisa_status_string(pisa.PISA_ERR_WORKSPACE) == "workspace too small"


def test_fused_schedule_needs_no_workspace():
    assert pisa.pisa_select_workspace_bytes(_good(schedule=pisa.PISA_SCHEDULE_FUSED)) == 0


def test_pyramid_append_validates_n_old():
    p = _good()
    lib = pisa.library()
    for bad in (-1, p.N + 1):
        assert lib.pisa_pyramid_append(ctypes.byref(p), FAKE, FAKE, bad, None) == pisa.PISA_ERR_INVALID_ARG
        assert "n_old" in pisa.pisa_last_error()
    assert lib.pisa_pyramid_append(ctypes.byref(p), None, FAKE, 0, None) == pisa.PISA_ERR_INVALID_ARG
    # n_old == N: nothing to do, nothing launched
    assert lib.pisa_pyramid_append(ctypes.byref(p), FAKE, FAKE, p.N, None) == pisa.PISA_OK


def test_capacity_layout():
    """With Ncap > N the pyramid is laid out for Ncap tokens; N's levels sit at
    the capacity offsets and the buffer size follows Ncap."""
    p = _good(N=1000, Ncap=4096, C=64)
    q = _good(N=4096, C=64)
    L = pisa.library()
    offs = (ctypes.c_int64 * 32)()
    R = ctypes.c_int64()
    Lp = L.pisa_pyramid_layout(ctypes.byref(p), offs, ctypes.byref(R))
    offs_q = (ctypes.c_int64 * 32)()
    Rq = ctypes.c_int64()
    Lq = L.pisa_pyramid_layout(ctypes.byref(q), offs_q, ctypes.byref(Rq))
    assert Lp == 5 and Lq == 7  # 16 and 64 leaf blocks with fanout 2
    assert R.value == Rq.value == 64 + 32 + 16 + 8 + 4 + 2
    assert list(offs[:Lp - 1]) == list(offs_q[:Lp - 1]) == [0, 64, 96, 112]
    assert offs[Lp - 1] == R.value  # the root is not stored
    assert pisa.pisa_pyramid_bytes(p) == pisa.pisa_pyramid_bytes(q)



def test_selection_quality_validates_before_launch():
    p = _good()
    lib = pisa.library()
    n = 37
    need = pisa.pisa_quality_workspace_bytes(p, n)
    M1 = -(-p.N // p.C)
    assert need == p.B * p.Hkv * n * (p.H // p.Hkv) * M1 * 4
    assert pisa.pisa_quality_workspace_bytes(p, 0) == 0

    def call(pp=p, rows=FAKE, n_rows=n, metrics=FAKE, ws=FAKE, nb=need):
        return lib.pisa_selection_quality(ctypes.byref(pp), FAKE, FAKE, FAKE, rows, n_rows, metrics, None, ws, nb,
                                          None)
    assert call(rows=None) == pisa.PISA_ERR_INVALID_ARG and "rows" in pisa.pisa_last_error()
    assert call(metrics=None) == pisa.PISA_ERR_INVALID_ARG
    assert call(n_rows=0) == pisa.PISA_ERR_INVALID_ARG
    assert call(nb=need - 1) == pisa.PISA_ERR_WORKSPACE
    assert call(pp=_good(dtype="f32")) == pisa.PISA_ERR_UNSUPPORTED


def test_attention_backward_validates_before_launch():
    p = _good()
    lib = pisa.library()
    need = pisa.pisa_attn_bwd_workspace_bytes(p)
    assert need > 0
    args = [FAKE] * 10

    def call(pp=p, args=args, ws=FAKE, nb=need):
        return lib.pisa_sparse_attn_bwd(ctypes.byref(pp), *args, ws, nb, None)
    for i, name in enumerate(["q", "k", "v", "block_idx", "o", "lse", "d_o", "dq", "dk", "dv"]):
        bad = list(args)
        bad[i] = None
        assert call(args=bad) == pisa.PISA_ERR_INVALID_ARG, name
        assert name in pisa.pisa_last_error()
    assert call(nb=need - 1) == pisa.PISA_ERR_WORKSPACE
    assert call(pp=_good(dtype="f32")) == pisa.PISA_ERR_UNSUPPORTED
    assert pisa.pisa_attn_bwd_workspace_bytes(_good(dtype="f32")) == 0


# Decode cache capacity (App. B "Decode cache": each level grows by a fixed
# fraction when more room is needed).
@pytest.mark.parametrize("C", [32, 64, 128])
def test_cache_capacity_rule(C):
    assert pisa.pisa_cache_capacity(1000, 1000, C) == 1000      # fits: unchanged
    assert pisa.pisa_cache_capacity(1000, 10, C) == 1000
    for cap, need in [(0, 1), (0, 777), (512, 513), (768, 769), (4096, 9000), (1000, 1001)]:
        got = pisa.pisa_cache_capacity(cap, need, C)
        assert got % C == 0 and got >= need and got >= cap + (cap + 1) // 2, (cap, need, got)
        assert got - C < max(need, cap + (cap + 1) // 2), (cap, need, got)   # the smallest such multiple


def test_cache_capacity_grows_geometrically():
    """Streaming one token at a time from 1000 to 2^21 tokens: each growth
    multiplies the capacity by at least 3/2, so there are O(log N) of them
    (about 1.7 per doubling) and the rows copied over all growths stay below
    three times the final length (a geometric series)."""
    C, cap, n = 64, 1024, 1000
    growths, copied = 0, 0
    while n < (1 << 21):
        n += 1
        if n > cap:
            new = pisa.pisa_cache_capacity(cap, n, C)
            assert new >= 1.5 * cap
            copied += n - 1           # the rows that move
            cap = new
            growths += 1
    assert growths <= math.ceil(math.log((1 << 21) / 1024, 1.5)) + 1
    assert copied < 3 * (1 << 21)


def test_cache_capacity_limits():
    C = 64
    top = 65535 * C
    assert pisa.pisa_cache_capacity(top - 10, top - 5, C) == top          # clamped, still holds need
    assert pisa.pisa_cache_capacity(50000 * C, 50000 * C + 1, C) == top     # 3/2 would pass the limit
    lib = pisa.library()
    assert lib.pisa_cache_capacity(top, top + 1, C) == pisa.PISA_ERR_UNSUPPORTED
    assert lib.pisa_cache_capacity(-1, 5, C) == pisa.PISA_ERR_INVALID_ARG
    assert lib.pisa_cache_capacity(5, 0, C) == pisa.PISA_ERR_INVALID_ARG
    with pytest.raises(pisa.PisaError):
        pisa.pisa_cache_capacity(top, top + 1, C)


def test_cache_grow_validates_before_launch():
    p = _good(N=1000, Ncap=1024, C=64)
    lib = pisa.library()
    big = FAKE * 64

    def call(new_cap=1536, po=FAKE, pn=big, ko=None, kn=None, vo=None, vn=None, pp=p):
        return lib.pisa_cache_grow(ctypes.byref(pp), new_cap, po, pn, ko, kn, vo, vn, None)
    assert call(new_cap=1000) == pisa.PISA_ERR_INVALID_ARG and "capacity" in pisa.pisa_last_error()
    assert call(new_cap=65536 * 64) == pisa.PISA_ERR_UNSUPPORTED
    assert call(pn=FAKE + 4096) == pisa.PISA_ERR_INVALID_ARG and "overlap" in pisa.pisa_last_error()
    assert call(po=None) == pisa.PISA_ERR_INVALID_ARG
    assert call(ko=big * 2) == pisa.PISA_ERR_INVALID_ARG            # keys without the other three pointers
    assert call(ko=big * 2, kn=big * 3, vo=big * 4, vn=big * 3 + 4096) == pisa.PISA_ERR_INVALID_ARG  # k_new, v_new overlap
    assert call(pp=_good(d=96)) == pisa.PISA_ERR_UNSUPPORTED


def test_union_threshold_knob_returns_previous_value():
    prev = pisa.pisa_attn_union_min_tiles(5)
    try:
        assert prev == 1024  # the library's default
        assert pisa.pisa_attn_union_min_tiles(-7) == 5
        assert pisa.pisa_attn_union_min_tiles(0) == -1  # any negative value means off
        assert pisa.pisa_attn_union_min_tiles(prev) == 0
    finally:
        pisa.pisa_attn_union_min_tiles(prev)
