"""Row-tile union attention against the oracle, through the C ABI.

On the block-centric attention path, a tile of T = 256 / G consecutive query
rows of one (batch, KV head) whose selections together name at most
min(3K, 256) distinct leaf blocks is attended whole by the row-tile union
kernel; the other tiles go through the block-centric kernels.  The index
lists here are built on the host so that tiles of both kinds alternate:
windows of neighbouring blocks (a small union) and random blocks (a large
one), with padding, entries past the last block and (causal) future blocks
planted in both, rows of one tile that share only part of their lists, and a
tile whose rows select nothing.  Checks: o within 2e-2 max-abs and lse within
1e-3 of the oracle on every row of the first tiles and on sampled rows
elsewhere (lse = -inf where a row attends no token), and, white-box, that the
per-tile flags the kernel leaves at the end of the workspace are exactly the
tiles whose union fits, listed in ascending order with their count.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2609_31093_amd import inputs
from tests.helpers import dev

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2609_31093_amd import pisa
else:
    pisa = None

CASES = {
    # name: (B, H, Hkv, Nq, N, d, C, K, causal)
    "g1-c32-d128-causal": (1, 2, 2, 3000, 3000, 128, 32, 16, 1),
    "g2-c64-d64-ragged": (2, 4, 2, 2085, 2085, 64, 64, 6, 1),
    "g4-c128-d128": (1, 8, 2, 6000, 6000, 128, 128, 8, 1),
    "g8-c96-d64-suffix": (1, 16, 2, 2500, 4000, 64, 96, 5, 1),
    "g16-c64-d128-noncausal": (1, 32, 2, 2500, 2500, 128, 64, 6, 0),
    "g4-k40-causal": (1, 8, 2, 5000, 5000, 64, 32, 40, 1),
    "g2-k48-noncausal-suffix": (1, 4, 2, 3000, 8000, 64, 32, 48, 0),
}


def _lists(B, Hkv, Nq, N, C, K, causal, T, seed):
    """Index lists [B, Hkv, Nq, K]: even tiles windows, odd tiles random."""
    r = np.random.default_rng(seed)
    M1 = -(-N // C)
    idx = np.full((B, Hkv, Nq, K), -1, dtype=np.int32)
    for b in range(B):
        for h in range(Hkv):
            for row in range(Nq):
                t = N - Nq + row
                c = t // C
                tile = row // T
                hi = c if causal else M1 - 1
                if tile == 2:
                    continue  # every row of this tile selects nothing
                if tile % 2 == 0:
                    if causal:
                        win = [0] + [x for x in range(c, max(c - K, 0), -1)]
                    else:
                        lo = max(0, min(c - K // 2, M1 - K))
                        win = list(range(lo, min(lo + K, M1)))
                    win = list(dict.fromkeys(win))[:K]
                else:
                    win = list(r.choice(hi + 1, size=min(K, hi + 1), replace=False))
                row_list = np.full(K, -1, dtype=np.int64)
                row_list[:len(win)] = win
                r.shuffle(row_list)
                kind = row % 11
                if kind == 1:
                    row_list[0] = -1
                elif kind == 3:
                    row_list[-1] = M1 + row % 7
                elif kind == 5:
                    row_list[-1] = (1 << 30) - row
                elif kind == 7 and causal and c + 1 < M1:
                    row_list[-1] = min(c + 1 + row % 3, M1 - 1)
                if len(set(int(x) for x in row_list if x >= 0)) < (row_list >= 0).sum():
                    row_list[-1] = -1  # keep the entries distinct
                idx[b, h, row] = row_list
    return idx


def _expected_flags(idx, N, C, K, T):
    M1 = -(-N // C)
    B, Hkv, Nq, _ = idx.shape
    tiles = -(-Nq // T)
    want = np.zeros((B * Hkv, tiles), dtype=np.uint8)
    for bh in range(B * Hkv):
        lst = idx.reshape(B * Hkv, Nq, K)[bh]
        for tl in range(tiles):
            blk = lst[tl * T:(tl + 1) * T].ravel()
            u = np.unique(blk[(blk >= 0) & (blk < M1)])
            want[bh, tl] = len(u) <= min(3 * K, 256)
    return want


@pytest.fixture
def union_min_tiles():
    """Sets the union threshold for one test and restores it afterwards."""
    prev = []

    def set_(n):
        r = pisa.pisa_attn_union_min_tiles(n)
        if not prev:
            prev.append(r)

    yield set_
    if prev:
        pisa.pisa_attn_union_min_tiles(prev[0])


@pytest.mark.parametrize("name", list(CASES))
def test_union_tiles_match_oracle(name, union_min_tiles):
    B, H, Hkv, Nq, N, d, C, K, causal = CASES[name]
    print("case", name, CASES[name], flush=True)
    union_min_tiles(0)  # these problems are smaller than the default threshold
    G = H // Hkv
    T = 256 // G
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=23)
    q, k, v = dev(x["q"], "bf16"), dev(x["k"], "bf16"), dev(x["v"], "bf16")
    idx_np = _lists(B, Hkv, Nq, N, C, K, bool(causal), T, seed=5)
    want_flags = _expected_flags(idx_np, N, C, K, T)
    others = [t for t in range(want_flags.shape[1]) if t != 2]
    assert want_flags[:, others].any() and not want_flags.all(), "the lists must give tiles of both kinds"
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, causal, "bf16")
    nb = pisa.pisa_attn_workspace_bytes(p)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((B, H, Nq), dtype=torch.float32, device="cuda")
    pisa.pisa_sparse_attn_fwd(p, q, k, v, torch.from_numpy(idx_np).cuda(), o, lse, ws, nb)
    torch.cuda.synchronize()
    # the workspace ends with the per-tile flags and then the flagged tiles'
    # ids followed by their count (256-byte aligned regions)
    nflag = B * Hkv * (-(-Nq // T))
    al = lambda n: (n + 255) // 256 * 256
    lstart = nb - al((nflag + 1) * 4)
    start = lstart - al(nflag)
    got_flags = ws[start:start + nflag].cpu().numpy().reshape(want_flags.shape)
    assert np.array_equal(got_flags, want_flags)
    tl = ws[lstart:lstart + (nflag + 1) * 4].cpu().view(torch.int32).numpy()
    ids = np.flatnonzero(want_flags.ravel())
    assert tl[nflag] == len(ids)
    assert np.array_equal(tl[:len(ids)], ids)
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([np.arange(min(Nq, 4 * T)), rng.choice(Nq, 96, replace=False), [Nq - 1]]))
    if G >= 8:
        rows = np.unique(np.concatenate([np.arange(min(Nq, 3 * T)), rng.choice(Nq, 40, replace=False), [Nq - 1]]))
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, bool(causal), rows=rows)
    got_o = o.float().cpu().numpy()[:, :, rows]
    got_lse = lse.cpu().numpy()[:, :, rows]
    assert np.abs(got_o - want_o).max() <= 2e-2
    empty = np.isneginf(want_lse)
    assert np.array_equal(np.isneginf(got_lse), empty)
    assert np.abs(got_lse[~empty] - want_lse[~empty]).max() <= 1e-3
    assert not np.any(got_o[empty])


@pytest.mark.parametrize("mode", ["default-threshold", "off"])
def test_union_threshold_and_off(mode, union_min_tiles):
    """Below the threshold (default 1024 qualifying tiles) the flags are
    cleared and the count is zero, so the block-centric kernels take every
    row; with the path off nothing is planned.  Results match the oracle and,
    to the last bit, the union path's where no union tile is involved."""
    name = "g4-k40-causal"
    B, H, Hkv, Nq, N, d, C, K, causal = CASES[name]
    print("case", name, mode, flush=True)
    G = H // Hkv
    T = 256 // G
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=23)
    q, k, v = dev(x["q"], "bf16"), dev(x["k"], "bf16"), dev(x["v"], "bf16")
    idx_np = _lists(B, Hkv, Nq, N, C, K, bool(causal), T, seed=5)
    want_flags = _expected_flags(idx_np, N, C, K, T)
    assert 0 < want_flags.sum() < 1024
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, 2, K, causal, "bf16")
    nb = pisa.pisa_attn_workspace_bytes(p)
    idx = torch.from_numpy(idx_np).cuda()

    def run(n):
        union_min_tiles(n)
        ws = torch.full((nb,), 0xAB, dtype=torch.uint8, device="cuda")
        o = torch.empty_like(q)
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device="cuda")
        pisa.pisa_sparse_attn_fwd(p, q, k, v, idx, o, lse, ws, nb)
        torch.cuda.synchronize()
        return o, lse, ws

    o_u, lse_u, _ = run(0)
    o, lse, ws = run(1024 if mode == "default-threshold" else -1)
    nflag = B * Hkv * (-(-Nq // T))
    al = lambda n: (n + 255) // 256 * 256
    lstart = nb - al((nflag + 1) * 4)
    start = lstart - al(nflag)
    if mode == "default-threshold":
        assert not ws[start:start + nflag].cpu().numpy().any()
        assert ws[lstart + 4 * nflag:lstart + 4 * nflag + 4].cpu().view(torch.int32).item() == 0
    else:
        assert (ws[start:start + nflag].cpu().numpy() == 0xAB).all()
    # rows of tiles the union kernel did not take come out identical
    for bh in range(B * Hkv):
        b, h = divmod(bh, Hkv)
        rows_blk = torch.from_numpy(np.flatnonzero(~np.repeat(want_flags[bh], T)[:Nq].astype(bool))).cuda()
        heads = slice(h * G, (h + 1) * G)
        assert torch.equal(o[b, heads][:, rows_blk], o_u[b, heads][:, rows_blk])
        assert torch.equal(lse[b, heads][:, rows_blk], lse_u[b, heads][:, rows_blk])
    rng = np.random.default_rng(2)
    rows = np.unique(np.concatenate([np.arange(min(Nq, 4 * T)), rng.choice(Nq, 96, replace=False), [Nq - 1]]))
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, bool(causal), rows=rows)
    got_o = o.float().cpu().numpy()[:, :, rows]
    got_lse = lse.cpu().numpy()[:, :, rows]
    assert np.abs(got_o - want_o).max() <= 2e-2
    empty = np.isneginf(want_lse)
    assert np.array_equal(np.isneginf(got_lse), empty)
    assert np.abs(got_lse[~empty] - want_lse[~empty]).max() <= 1e-3


def test_forced_block_tiles_across_row_chunks():
    """8 heads per KV head with a budget of 64: the per-slot partials of
    60000 rows exceed the 6 GiB the block-centric path holds at once, so the
    attention runs in three row chunks (whole 256-row tiles each) and every
    chunk's forced-block tiles merge 61 far partials per (row, head) (no
    separate tail merge).  The selection is the library's own; rows on both
    sides of each chunk boundary and random rows against the oracle."""
    B, H, Hkv, d, C, g, K = 1, 16, 2, 128, 64, 2, 64
    N = Nq = 60000
    G = H // Hkv
    per_row = B * Hkv * K * G * (2 * d + 4)
    ch = (6 << 30) // per_row // 256 * 256
    assert ch < Nq < 3 * ch
    print("case chunks", ch, flush=True)
    x = inputs.random_qkv(B, H, Hkv, Nq, N, d, "bf16", seed=29)
    q, k, v = dev(x["q"], "bf16"), dev(x["k"], "bf16"), dev(x["v"], "bf16")
    p = pisa.make_problem(B, H, Hkv, Nq, N, d, C, g, K, 1, "bf16")
    idx = pisa.select(p, q, k, pisa.build_pyramid(p, k))
    o, lse = pisa.sparse_attn_fwd(p, q, k, v, idx)
    torch.cuda.synchronize()
    idx_np = idx.cpu().numpy()
    rng = np.random.default_rng(4)
    rows = np.unique(np.concatenate([[0, 1, ch - 1, ch, 2 * ch - 1, 2 * ch, Nq - 1],
                                     rng.choice(Nq, 25, replace=False)]))
    want_o, want_lse = O.sparse_attention(x["q"], x["k"], x["v"], idx_np[:, :, rows], C, True, rows=rows)
    got_o = o.float().cpu().numpy()[:, :, rows]
    got_lse = lse.cpu().numpy()[:, :, rows]
    assert np.abs(got_o - want_o).max() <= 2e-2
    assert np.abs(got_lse - want_lse).max() <= 1e-3
