"""Shared helpers of the GPU parity tests: device upload, oracle comparison."""
import numpy as np
import torch


def dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t
    return t.to("cuda")


def check_selection_valid(idx: np.ndarray, N: int, Nq: int, C: int, K: int, causal: bool):
    """Properties every correct selection has: ascending unique in-range indices,
    the forced blocks present, and min(K, #eligible) entries."""
    B, Hkv, R, _ = idx.shape
    M1 = -(-N // C)
    for r in range(R):
        t = N - Nq + r
        c = t // C
        elig = c + 1 if causal else M1
        want_n = min(K, elig)
        for b in range(B):
            for h in range(Hkv):
                row = idx[b, h, r]
                sel = row[row >= 0]
                assert len(sel) == want_n, (b, h, r, row)
                assert np.all(row[want_n:] == -1)
                assert np.all(np.diff(sel) > 0)
                assert sel.min() >= 0 and sel.max() < (c + 1 if causal else M1)
                if causal:
                    for f in {0, c, max(c - 1, 0)}:
                        assert f in sel, (r, f, sel)


def compare_selection(gpu_idx: np.ndarray, ora_idx: np.ndarray, gap: np.ndarray, tol: float = 1e-3):
    """Indices must agree on every decisive row (oracle margin > tol).  Returns
    statistics of the near-tie rows, which are reported, not asserted."""
    gpu_idx = np.asarray(gpu_idx, dtype=np.int64)
    diff = (gpu_idx != ora_idx).any(axis=-1)
    decisive = gap > tol
    bad = np.argwhere(diff & decisive)
    assert bad.size == 0, (f"{len(bad)} decisive rows differ; first {bad[:5].tolist()}: "
                           f"gpu {gpu_idx[tuple(bad[0])].tolist()} oracle {ora_idx[tuple(bad[0])].tolist()} "
                           f"gap {gap[tuple(bad[0])]}")
    near = ~decisive
    return {"rows": int(diff.size), "decisive": int(decisive.sum()), "near_tie": int(near.sum()),
            "near_tie_differ": int((diff & near).sum()), "exact_tie": int((gap == 0).sum()),
            "exact_tie_differ": int((diff & (gap == 0)).sum())}
