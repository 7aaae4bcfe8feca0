"""Seeded synthetic inputs for the packed-cache path.

This module only draws random numbers and shapes them like the attention
inputs of the workloads the paper measures (Qwen2.5-3B / Llama-3.1-8B shaped
heads, d_h = 128).  It holds none of the method's arithmetic: no scores, no
allocation, no quantization, no attention.  Both the HIP path (through the
tests and the benchmark) and the CPU oracle consume what it produces.

Recipe (one generator stream per purpose, so any piece can be regenerated):

* ``numpy.random.default_rng([seed, layer, kv_head, kind, chunk])`` with kind
  0 energy profile, 1 calibration queries, 2 calibration keys, 3 keys,
  4 values, 5 decode queries, 6 ragged lengths, 7 rotations.
* Energy profile per (layer, KV head): sigma_i = exp(N(0, 1)) for each of the
  L = d_h / 2 RoPE blocks, and three distinct blocks scaled by 8 (outliers).
* Keys: pre-RoPE block i ~ N(0, sigma_i^2 I_2) on dims (i, i + d_h/2), then the
  rotary embedding at the token's position (angles in float64).
* Values ~ N(0, 1); queries ~ N(0, 1) per query head, rotary-embedded at the
  decode position.
* Rotations: Haar-distributed orthogonal matrices (Gaussian matrix, Householder
  QR in float64, column signs fixed so that diag(R) > 0), rounded to float32.
  One matrix per (stream, dimension): K uses d = 2, 4, ..., d_h and V uses d_h.
* Storage precision: float32, or bfloat16 (round to nearest even) stored in
  float32 arrays whose values are exactly representable in bfloat16.
"""
from __future__ import annotations

import numpy as np

KIND_PROFILE, KIND_QCAL, KIND_KCAL, KIND_K, KIND_V, KIND_Q, KIND_LENS, KIND_ROT = range(8)


def rng(seed: int, layer: int, head: int, kind: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(layer), int(head), int(kind), int(chunk)])


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def cast(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "fp32":
        return x
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(dtype)


def sigma_profile(seed: int, layer: int, head: int, n_blocks: int = 64,
                  n_outliers: int = 3, outlier_scale: float = 8.0) -> np.ndarray:
    g = rng(seed, layer, head, KIND_PROFILE)
    sigma = np.exp(g.standard_normal(n_blocks))
    idx = g.choice(n_blocks, size=n_outliers, replace=False)
    sigma[idx] *= outlier_scale
    return sigma


def _rotary(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary embedding with half-split pairs (i, i + d/2); x [..., n, d], pos [n]."""
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def keys(seed, layer, head, t0, n, sigma, base, d_h=128, pre_rope=False, chunk=None):
    """Keys for positions t0 .. t0+n-1 of one (layer, KV head), float64 [n, d_h]."""
    g = rng(seed, layer, head, KIND_K, t0 if chunk is None else chunk)
    half = d_h // 2
    z = g.standard_normal((n, d_h))
    scale = np.concatenate([sigma, sigma])[None, :half * 2]
    k = z * scale
    if pre_rope:
        return k
    return _rotary(k, np.arange(t0, t0 + n), base)


def values(seed, layer, head, t0, n, d_h=128, chunk=None):
    g = rng(seed, layer, head, KIND_V, t0 if chunk is None else chunk)
    return g.standard_normal((n, d_h))


def queries(seed, layer, head, pos, group, base, d_h=128, step=0):
    """Post-RoPE decode queries of the `group` query heads reading KV head `head`."""
    g = rng(seed, layer, head, KIND_Q, step)
    q = g.standard_normal((group, d_h))
    return _rotary(q[:, None, :], np.array([pos]), base)[:, 0, :]


def calibration(seed, layer, head, n_cal, group, sigma, d_h=128):
    """Pre-RoPE calibration activations: q [n_cal, group, d_h], k [n_cal, d_h]."""
    gq = rng(seed, layer, head, KIND_QCAL)
    gk = rng(seed, layer, head, KIND_KCAL)
    q = gq.standard_normal((n_cal, group, d_h))
    k = gk.standard_normal((n_cal, d_h)) * np.concatenate([sigma, sigma])[None, :]
    return q, k


def haar_orthogonal(d: int, g: np.random.Generator) -> np.ndarray:
    a = g.standard_normal((d, d))
    qm, r = np.linalg.qr(a)
    qm = qm * np.sign(np.diag(r))[None, :]
    return qm


def rotations(seed: int, d_h: int = 128):
    """K rotations for every even d <= d_h and the V rotation, all float32.

    Returns (rot_k, rot_v): rot_k is a dict d -> [d, d]; rot_v is [d_h, d_h].
    """
    rot_k = {}
    for d in range(2, d_h + 1, 2):
        rot_k[d] = haar_orthogonal(d, rng(seed, 0, 0, KIND_ROT, d)).astype(np.float32)
    rot_v = haar_orthogonal(d_h, rng(seed, 1, 0, KIND_ROT, d_h)).astype(np.float32)
    return rot_k, rot_v


def flat_rot_k(rot_k: dict, d_h: int = 128) -> np.ndarray:
    """Concatenate the K rotations for d = 2, 4, ..., d_h (row-major each)."""
    return np.concatenate([rot_k[d].reshape(-1) for d in range(2, d_h + 1, 2)]).astype(np.float32)


def ragged_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    g = rng(seed, 0, 0, KIND_LENS)
    return g.integers(lo, hi + 1, size=batch).astype(np.int64)


# --------------------------------------------------------------------------
# Device-side generator for the long-context workloads (same recipe; the
# stream is torch's CUDA generator seeded per (seed, layer, kind)).
# --------------------------------------------------------------------------

def torch_layer_kv(seed: int, layer: int, n: int, sigma: np.ndarray, base: float, t0: int = 0,
                   device="cuda", dtype=None):
    """Keys and values of every KV head of one layer for positions t0..t0+n-1.

    sigma: [n_kv, 64] block profile.  Returns (k, v) [n, n_kv, 128] in `dtype`
    (default bfloat16); keys rotary-embedded with float64 angles."""
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    n_kv = sigma.shape[0]
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + int(layer) * 101 + 3)
    z = torch.randn((n, n_kv, 128), generator=g, device=device, dtype=torch.float32)
    sc = torch.from_numpy(np.concatenate([sigma, sigma], axis=1).astype(np.float32)).to(device)
    k = z * sc[None]
    k = _torch_rotary(k, torch.arange(t0, t0 + n, device=device, dtype=torch.float64), base)
    g.manual_seed(int(seed) * 1000003 + int(layer) * 101 + 4)
    v = torch.randn((n, n_kv, 128), generator=g, device=device, dtype=torch.float32)
    return k.to(dtype), v.to(dtype)


def torch_queries(seed: int, layer: int, n_q: int, pos, base: float, device="cuda", dtype=None):
    """Decode queries [len(pos), n_q, 128] at positions `pos` (one per step)."""
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    pos = torch.as_tensor(pos, dtype=torch.float64, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + int(layer) * 101 + 5)
    q = torch.randn((pos.numel(), n_q, 128), generator=g, device=device, dtype=torch.float32)
    return _torch_rotary(q, pos, base).to(dtype)


def _torch_rotary(x, pos, base):
    import torch
    inv = base ** (-2.0 * torch.arange(64, dtype=torch.float64, device=x.device) / 128)
    ang = pos[:, None] * inv[None, :]
    c = torch.cos(ang).to(torch.float32)[:, None, :]
    s = torch.sin(ang).to(torch.float32)[:, None, :]
    a, b = x[..., :64], x[..., 64:]
    return torch.cat([a * c - b * s, a * s + b * c], dim=-1)
