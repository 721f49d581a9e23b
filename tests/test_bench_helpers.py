"""bench.py's replica of the row-tile union rule (union_rows), on the CPU,
against a brute-force count of each tile's distinct blocks: the tiles it
reports are exactly those of 256 / G rows naming at most min(3K, 256) valid
blocks, the threshold and the head-group restriction apply, and its staging
count is the sum of the taken tiles' unions."""
import numpy as np
import pytest
import torch

import bench


def _brute(idx, N, C, K, G):
    B, Hkv, Nq, _ = idx.shape
    M1 = -(-N // C)
    T = 256 // G
    tiles = -(-Nq // T)
    ok = np.zeros((B * Hkv, tiles), dtype=bool)
    size = np.zeros((B * Hkv, tiles), dtype=np.int64)
    flat = idx.reshape(B * Hkv, Nq, K)
    for bh in range(B * Hkv):
        for t in range(tiles):
            blk = flat[bh, t * T:(t + 1) * T].ravel()
            u = np.unique(blk[(blk >= 0) & (blk < M1)])
            size[bh, t] = len(u)
            ok[bh, t] = len(u) <= min(3 * K, 256)
    return ok, size, T


@pytest.mark.parametrize("G", [1, 4, 16])
def test_union_rows_match_brute_force(G):
    rng = np.random.default_rng(G)
    B, Hkv, N, C, K, d = 1, 2, 5000, 32, 6, 64
    Nq = N
    M1 = -(-N // C)
    idx = np.full((B, Hkv, Nq, K), -1, dtype=np.int64)
    for row in range(Nq):
        c = row // C
        if (row // (256 // G)) % 2 == 0:  # windows: small unions
            win = list(range(max(0, c - K + 1), c + 1))
        else:  # random blocks: large unions
            win = list(rng.choice(c + 1, size=min(K, c + 1), replace=False))
        idx[:, :, row, :len(win)] = win
    idx[0, 0, 7, 0] = M1 + 3  # past the last block: padding
    w = dict(B=B, H=Hkv * G, Hkv=Hkv, N=N, Nq=Nq, d=d, C=C, K=K, dtype="bf16", causal=1)
    ok, size, T = _brute(idx, N, C, K, G)
    got = bench.union_rows(torch.from_numpy(idx), w, 0)
    assert got is not None
    rows, stagings = got
    want_rows = np.repeat(ok, T, axis=1)[:, :Nq].reshape(B, Hkv, Nq)
    assert np.array_equal(rows.numpy(), want_rows)
    assert stagings == int((size * ok).sum())
    # fewer qualifying tiles than the threshold: nothing taken; off: nothing taken
    assert bench.union_rows(torch.from_numpy(idx), w, int(ok.sum()) + 1) is None
    assert bench.union_rows(torch.from_numpy(idx), w, -1) is None
    # 3 heads per KV head: no union kernel
    assert bench.union_rows(torch.from_numpy(idx), dict(w, H=Hkv * 3), 0) is None
