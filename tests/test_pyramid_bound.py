"""The per-node float32 error bound of the pyramid (tests/helpers.py
pyramid_error_bound), on the CPU: float32 emulations of the mean pyramid in
three summation orders (sequential, pairwise tree, reversed) stay within it on
every element, for full and ragged last blocks, fan-outs 2 and 4 and block
sizes with and without an exact reciprocal; and it is tighter than the single
global bound (C + L g) 2^-24 max|k| it replaces."""
import numpy as np
import pytest

import oracle as O
from tests.helpers import pyramid_error_bound


def _f32_mean(x, order):
    x = x.astype(np.float32)
    if order == "seq":
        s = np.zeros(x.shape[1:], dtype=np.float32)
        for r in x:
            s = np.float32(s + r)
    elif order == "rev":
        s = np.zeros(x.shape[1:], dtype=np.float32)
        for r in x[::-1]:
            s = np.float32(s + r)
    else:  # pairwise tree
        v = list(x)
        while len(v) > 1:
            v = [np.float32(v[i] + v[i + 1]) if i + 1 < len(v) else v[i] for i in range(0, len(v), 2)]
        s = v[0]
    return np.float32(s * np.float32(1.0 / x.shape[0]))


def _f32_pyramid(k, C, g, order):
    N, d = k.shape
    M = O.level_sizes(N, C, g)
    lv = [np.stack([_f32_mean(k[i * C:min((i + 1) * C, N)], order) for i in range(M[0])])]
    for m in M[1:]:
        lv.append(np.stack([_f32_mean(lv[-1][i * g:min((i + 1) * g, lv[-1].shape[0])], order) for i in range(m)]))
    return O.pyramid_rows([x.astype(np.float64) for x in lv])


@pytest.mark.parametrize("N,C,g", [(4096, 64, 2), (3000, 96, 2), (5000, 32, 4), (2085, 64, 4)])
@pytest.mark.parametrize("order", ["seq", "tree", "rev"])
def test_float32_pyramid_within_bound(N, C, g, order):
    rng = np.random.default_rng(N + C + g)
    k = (rng.standard_normal((1, 1, N, 16)) * 3.0 + 0.5).astype(np.float32)
    want = O.pyramid(k, C, g)
    got = _f32_pyramid(k[0, 0], C, g, order)
    bound = pyramid_error_bound(k, C, g)
    err = np.abs(got - want[0, 0])
    assert np.all(err <= bound[0, 0]), float((err - bound[0, 0]).max())
    # tighter than the global bound, on every element
    L = len(O.level_sizes(N, C, g))
    assert bound.max() < (C + L * g) * 2.0 ** -24 * float(np.abs(k).max())
