"""Seeded synthetic inputs for the PISA hot path.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the method's arithmetic: the pyramid, the scores, the
selection and the attention live in the HIP library (and, independently, in
the CPU oracle used by the tests).

Workloads (B = batch, H = query heads, Hkv = KV heads, N = keys, Nq = query
rows, d = head dim, C = leaf block size, g = fan-out, K = block budget):

* ``tiny-fp32``    fp32, B=1, H=Hkv=2, N=4096, d=64, C=64, g=2, K=4;
                   q, k, v i.i.d. N(0,1).
* ``gqa-32k``      bf16, B=1, H=16, Hkv=4, N=32768, d=128, C=64, g=2, K=16;
                   q, k, v i.i.d. N(0,1), q multiplied by 1/sqrt(128) before
                   rounding.
* ``needles-128k`` bf16, B=1, H=Hkv=8, N=131072, d=128, C=64, g=2, K=16;
                   k, v i.i.d. N(0,1); 32 needle leaf blocks (drawn without
                   replacement from blocks 1..M-1) whose keys in every head
                   equal 4u for one seeded unit vector u; N/4 seeded query
                   positions (shared by all heads) set to u + 0.5 N(0, I).
* ``ar1-512k``     bf16, B=1, H=8, Hkv=2, N=524288, d=128, C=128, g=4, K=32;
                   q and k follow independent stationary AR(1) processes along
                   the sequence (rho = 0.999) per (head, dim); v i.i.d. N(0,1).
* ``decode-128k``  bf16, B=1, H=Hkv=8, N=131072, Nq=1, d=128, C=64, g=2,
                   K=16; k, v i.i.d. N(0,1); 64 single-token query steps.
* ``paper-sel-128k`` bf16, B=1, H=32, Hkv=2, N=131072, d=64, C=64, g=2, K=8
                   (the paper's block-selection benchmark shape); q, k, v
                   i.i.d. N(0,1).

Every (batch, head) slice of every tensor comes from its own stream
``np.random.default_rng(SeedSequence([seed, cfg_id, tensor_id, b, h]))`` in
float32 (needle positions and the needle direction from stream
``[seed, cfg_id, 3]``) and is then rounded to bfloat16 (round to nearest even)
when the workload is bf16.  The arrays returned are float32 holding the
exact stored values, so the GPU (which receives bf16) and the oracle (which
widens to float64) see identical numbers.
"""
from __future__ import annotations

import numpy as np

WORKLOADS = {
    "tiny-fp32": dict(cfg_id=1, B=1, H=2, Hkv=2, N=4096, Nq=None, d=64, C=64, g=2, K=4,
                      causal=1, dtype="f32", dist="iid"),
    "gqa-32k": dict(cfg_id=2, B=1, H=16, Hkv=4, N=32768, Nq=None, d=128, C=64, g=2, K=16,
                    causal=1, dtype="bf16", dist="iid_qscaled"),
    "needles-128k": dict(cfg_id=3, B=1, H=8, Hkv=8, N=131072, Nq=None, d=128, C=64, g=2, K=16,
                         causal=1, dtype="bf16", dist="needles"),
    "ar1-512k": dict(cfg_id=4, B=1, H=8, Hkv=2, N=524288, Nq=None, d=128, C=128, g=4, K=32,
                     causal=1, dtype="bf16", dist="ar1"),
    "decode-128k": dict(cfg_id=5, B=1, H=8, Hkv=8, N=131072, Nq=1, d=128, C=64, g=2, K=16,
                        causal=1, dtype="bf16", dist="iid", steps=64),
    # the shape of the paper's block-selection latency benchmark (App. B):
    # 32 query heads on 2 KV heads, d = 64, C = 64, K = 8, g = 2, random bf16 q and k
    "paper-sel-128k": dict(cfg_id=6, B=1, H=32, Hkv=2, N=131072, Nq=None, d=64, C=64, g=2, K=8,
                           causal=1, dtype="bf16", dist="iid"),
}

_Q, _K, _V, _AUX = 0, 1, 2, 3


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _rng(seed: int, cfg_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg_id, tensor_id]))


def _per_head(seed: int, cfg_id: int, tensor_id: int, shape, fill) -> np.ndarray:
    """Fill a [B, Hx, ...] float32 array one (b, h) slice at a time, each slice
    from its own stream SeedSequence([seed, cfg_id, tensor_id, b, h])."""
    from concurrent.futures import ThreadPoolExecutor

    out = np.empty(shape, dtype=np.float32)
    B, Hx = shape[0], shape[1]

    def one(i):
        b, h = divmod(i, Hx)
        rng = np.random.default_rng(np.random.SeedSequence([seed, cfg_id, tensor_id, b, h]))
        out[b, h] = fill(rng, shape[2:])

    with ThreadPoolExecutor(max_workers=max(1, min(16, B * Hx))) as ex:
        list(ex.map(one, range(B * Hx)))
    return out


def _normal_fill(rng, shape):
    return rng.standard_normal(size=shape, dtype=np.float32)


def _ar1_fill(rng, shape, rho: float = 0.999) -> np.ndarray:
    """Stationary AR(1) along axis -2: x_0 ~ N(0,1), x_t = rho x_{t-1} + sqrt(1-rho^2) e_t."""
    from scipy.signal import lfilter

    e = rng.standard_normal(size=shape)  # float64 for the recursion
    e[..., 0, :] /= np.sqrt(1.0 - rho * rho)  # so that x_0 = e_0 ~ N(0,1) after scaling below
    x = lfilter([1.0], [1.0, -rho], e, axis=-2) * np.sqrt(1.0 - rho * rho)
    return x.astype(np.float32)


def workload(name: str, **overrides) -> dict:
    """Return the shape dict of a named workload, with overrides (e.g. N=...)."""
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    w = dict(WORKLOADS[name])
    w.update(overrides)
    w["name"] = name
    if w.get("Nq") is None:
        w["Nq"] = w["N"]
    return w


def make_inputs(w: dict, seed: int = 0, step: int = 0, parts: str = "qkv") -> dict:
    """Draw q [B,H,Nq,d], k [B,Hkv,N,d], v [B,Hkv,N,d] for workload dict ``w``.

    ``step`` selects the query of a decode step (decode workloads draw a fresh
    query per step; k and v do not depend on it).  ``parts`` limits which
    tensors are returned for the i.i.d. workloads (e.g. "q" for later decode
    steps); the others always return all three.
    """
    B, H, Hkv, N, Nq, d, C = w["B"], w["H"], w["Hkv"], w["N"], w["Nq"], w["d"], w["C"]
    cid = w["cfg_id"]
    dist = w["dist"]
    qshape, kshape = (B, H, Nq, d), (B, Hkv, N, d)
    q_tid = _Q if step == 0 else 16 + step
    if dist in ("iid", "iid_qscaled"):
        q = _per_head(seed, cid, q_tid, qshape, _normal_fill)
        if dist == "iid_qscaled":
            q *= np.float32(1.0 / np.sqrt(d))
        if parts == "q":
            return {"q": round_to_bf16(q) if w["dtype"] == "bf16" else q}
        k = _per_head(seed, cid, _K, kshape, _normal_fill)
        v = _per_head(seed, cid, _V, kshape, _normal_fill)
    elif dist == "needles":
        rng_aux = _rng(seed, cid, _AUX)
        n = rng_aux.standard_normal(d)
        u = (n / np.linalg.norm(n)).astype(np.float32)
        M1 = -(-N // C)
        n_needles = min(32, max(0, M1 - 1))
        needle_blocks = np.sort(rng_aux.choice(np.arange(1, M1), size=n_needles, replace=False)) \
            if n_needles else np.zeros(0, dtype=np.int64)
        n_qpos = Nq // 4
        qpos = np.sort(rng_aux.choice(Nq, size=n_qpos, replace=False)) if n_qpos else np.zeros(0, np.int64)
        k = _per_head(seed, cid, _K, kshape, _normal_fill)
        for b in needle_blocks:
            k[:, :, b * C:min((b + 1) * C, N), :] = 4.0 * u
        q = _per_head(seed, cid, q_tid, qshape, _normal_fill)
        if n_qpos:
            noise = _per_head(seed, cid, _AUX + 10, (B, H, n_qpos, d), _normal_fill)
            q[:, :, qpos, :] = u + 0.5 * noise
        v = _per_head(seed, cid, _V, kshape, _normal_fill)
    elif dist == "ar1":
        q = _per_head(seed, cid, q_tid, qshape, _ar1_fill)
        k = _per_head(seed, cid, _K, kshape, _ar1_fill)
        v = _per_head(seed, cid, _V, kshape, _normal_fill)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    if w["dtype"] == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    return {"q": np.ascontiguousarray(q, np.float32),
            "k": np.ascontiguousarray(k, np.float32),
            "v": np.ascontiguousarray(v, np.float32)}


def needle_layout(w: dict, seed: int = 0) -> dict:
    """Needle block indices and needle query positions of a ``needles`` workload."""
    N, Nq, C, d, cid = w["N"], w["Nq"], w["C"], w["d"], w["cfg_id"]
    rng_aux = _rng(seed, cid, _AUX)
    n = rng_aux.standard_normal(d)
    M1 = -(-N // C)
    n_needles = min(32, max(0, M1 - 1))
    blocks = np.sort(rng_aux.choice(np.arange(1, M1), size=n_needles, replace=False))
    qpos = np.sort(rng_aux.choice(Nq, size=Nq // 4, replace=False))
    return {"u": (n / np.linalg.norm(n)).astype(np.float32), "blocks": blocks, "qpos": qpos}


def random_qkv(B: int, H: int, Hkv: int, Nq: int, N: int, d: int, dtype: str = "bf16",
               seed: int = 0, q_scale: float = 1.0) -> dict:
    """i.i.d. N(0,1) q, k, v of arbitrary shape (q times q_scale), rounded to dtype."""
    r = np.random.default_rng(np.random.SeedSequence([seed, 1000 + B, H, Hkv, Nq, N, d]))
    q = r.standard_normal((B, H, Nq, d), dtype=np.float32) * np.float32(q_scale)
    k = r.standard_normal((B, Hkv, N, d), dtype=np.float32)
    v = r.standard_normal((B, Hkv, N, d), dtype=np.float32)
    if dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    return {"q": q, "k": k, "v": v}
