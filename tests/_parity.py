"""Shared helpers of the GPU parity tests (not collected by pytest).

The HIP side runs through the C ABI binding; the oracle side runs the fp64
CPU oracle on the same seeded inputs.  Nothing from the HIP side is fed into
an oracle function: packed words coming back from the GPU are decoded by the
small test-local readers below.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from oracle import blockgtq_oracle as o
from paper_2606_24033_amd import blockgtq as bg
from paper_2606_24033_amd import synth

U = 2.0 ** -23  # twice the fp32 unit roundoff


# ------------------------------------------------------------------ readers

def read_fields(words: np.ndarray, widths) -> np.ndarray:
    """Codes of rows of LSB-first dense fields (test-local reader)."""
    w = words.astype(np.uint64)
    out = np.zeros((w.shape[0], len(widths)), dtype=np.int64)
    off = 0
    for p, b in enumerate(widths):
        lo = w[:, off // 32]
        hi = w[:, off // 32 + 1] if (off % 32 + b > 32) else np.zeros_like(lo)
        v = (lo | (hi << np.uint64(32))) >> np.uint64(off % 32)
        out[:, p] = (v & np.uint64((1 << int(b)) - 1)).astype(np.int64)
        off += int(b)
    return out


def read_value_codes(tiles: np.ndarray, b_v: int, n: int) -> np.ndarray:
    """tiles [n_tiles, 128, b_v] -> codes [n, 128] of tokens 0..n-1."""
    per_tile = tiles.reshape(tiles.shape[0], 128, b_v)
    out = np.zeros((n, 128), dtype=np.int64)
    for t in range(0, n, 32):
        m = min(32, n - t)
        out[t:t + m] = read_fields(per_tile[t // 32], [b_v] * 32)[:, :m].T
    return out


# ------------------------------------------------------------------ setup

@dataclass
class Setup:
    cfg: bg.Config
    seed: int
    base: float
    dtype: str
    bits: np.ndarray            # [n_layers, n_kv, 64] from the library
    bits_oracle: np.ndarray     # same, from the oracle
    sigma: dict = field(default_factory=dict)
    rot_k: dict = None
    rot_v: np.ndarray = None


def make_setup(seed, n_layers, batch, n_kv, group, capacity, k_budget, v_bits, base, dtype="bf16",
               n_cal=256, uniform=False):
    """uniform=True: every RoPE block at k_budget / 64 bits (the uniform
    TQ-MSE K layout, one K group) instead of the allocator's widths."""
    cfg = bg.Config(n_layers=n_layers, batch=batch, n_kv_heads=n_kv, group=group, capacity=capacity,
                    k_budget=k_budget, v_bits=v_bits,
                    in_dtype=bg.BGTQ_BF16 if dtype == "bf16" else bg.BGTQ_FP32)
    bits = np.zeros((n_layers, n_kv, 64), dtype=np.uint8)
    bits_o = np.zeros_like(bits)
    sig = {}
    for layer in range(n_layers):
        for h in range(n_kv):
            sig[layer, h] = synth.sigma_profile(seed, layer, h)
            qc, kc = synth.calibration(seed, layer, h, n_cal, group, sig[layer, h])
            qc, kc = qc.astype(np.float32), kc.astype(np.float32)
            if uniform:
                bits[layer, h] = bits_o[layer, h] = k_budget // 64
            else:
                bits[layer, h] = bg.blockgtq_allocate(bg.blockgtq_energy_scores(qc, kc), k_budget)[0]
                bits_o[layer, h] = o.allocate(o.energy_scores(qc, kc), k_budget)
    rot_k, rot_v = synth.rotations(seed)
    return Setup(cfg, seed, base, dtype, bits, bits_o, sig, rot_k, rot_v)


def keys_values(st: Setup, layer, head, t0, n):
    k = synth.cast(synth.keys(st.seed, layer, head, t0, n, st.sigma[layer, head], st.base), st.dtype)
    v = synth.cast(synth.values(st.seed, layer, head, t0, n), st.dtype)
    return k, v


# ------------------------------------------------------------------ oracle side

@dataclass
class OracleRows:
    kcodes: np.ndarray   # [n, 128] stream order
    widths: np.ndarray
    knorms: np.ndarray   # [n, n_g]
    kz: np.ndarray
    vcodes: np.ndarray
    vnorms: np.ndarray
    vz: np.ndarray
    kwords: np.ndarray
    kexact: np.ndarray   # [n, n_g] unrounded radii
    vexact: np.ndarray


def oracle_rows(st: Setup, layer, head, k, v) -> OracleRows:
    bits = st.bits_oracle[layer, head]
    kc, widths, kn, kz = o.quantize_keys(k, bits, st.rot_k)
    vc, vn, vz = o.quantize_values(v, st.rot_v, st.cfg.v_bits)
    kexact = np.stack([np.linalg.norm(np.asarray(k, np.float64)[:, dims], axis=1) for _, dims in o.groups(bits)], 1)
    vexact = np.linalg.norm(np.asarray(v, np.float64), axis=1)
    return OracleRows(kc, widths, kn, kz, vc, vn, vz, o.pack_key_rows(kc, widths), kexact, vexact)


# ------------------------------------------------------------------ comparisons

@dataclass
class Stats:
    codes: int = 0
    code_ties: int = 0
    norms: int = 0
    norm_ties: int = 0


def _tie_mask(z, widths, d_of_pos):
    """|z - nearest threshold| <= (d^1.5 + d |z|) 2^-23 for every position."""
    near = np.full(z.shape, np.inf)
    for b in np.unique(widths):
        cols = np.nonzero(widths == b)[0]
        _, thr = o.codebook(int(b))
        zz = z[:, cols]
        near[:, cols] = np.min(np.abs(zz[..., None] - thr[None, None, :]), axis=-1)
    d = d_of_pos[None, :].astype(np.float64)
    return near <= (d ** 1.5 + d * np.abs(z)) * U


def compare_codes(gpu_codes, ora_codes, z, widths, d_of_pos, stats: Stats, what=""):
    diff = gpu_codes != ora_codes
    stats.codes += gpu_codes.size
    if not diff.any():
        return
    tie = _tie_mask(z, np.asarray(widths), np.asarray(d_of_pos))
    bad = diff & ~(tie & (np.abs(gpu_codes - ora_codes) == 1))
    assert not bad.any(), f"{what}: {int(bad.sum())} code mismatches away from thresholds, first at {np.argwhere(bad)[:5]}"
    stats.code_ties += int(diff.sum())


def compare_norms(gpu16, ora16, exact, d, stats: Stats, what=""):
    gpu = np.asarray(gpu16, dtype=np.float64)
    diff = gpu != ora16
    stats.norms += gpu.size
    if not diff.any():
        return
    # allowed only next to an fp16 rounding midpoint of the exact radius
    lo, hi = np.minimum(gpu, ora16), np.maximum(gpu, ora16)
    mid = 0.5 * (lo + hi)
    tie = np.abs(exact - mid) <= d * U * exact * 4
    bad = diff & ~tie
    assert not bad.any(), f"{what}: {int(bad.sum())} norm mismatches, e.g. gpu={gpu[bad][:3]} oracle={ora16[bad][:3]}"
    stats.norm_ties += int(diff.sum())


def rel_err(out_gpu, out_ref):
    """max over rows of ||o_gpu - o_ref||_inf / ||o_ref||_inf."""
    num = np.max(np.abs(out_gpu - out_ref), axis=-1)
    den = np.max(np.abs(out_ref), axis=-1)
    return float(np.max(num / den))


def oracle_attention(st: Setup, layer, head, q, rows: OracleRows, ctx):
    bits = st.bits_oracle[layer, head]
    kh = o.dequantize_keys(rows.kcodes[:ctx], rows.knorms[:ctx], bits, st.rot_k)
    vh = o.dequantize_values(rows.vcodes[:ctx], rows.vnorms[:ctx], st.rot_v, st.cfg.v_bits)
    return o.attention(q, kh, vh)


def group_dims(bits):
    """d_g of every stream position (test-local)."""
    out = []
    for b in range(1, 9):
        n = int(np.sum(np.asarray(bits) == b))
        out += [2 * n] * (2 * n)
    return np.array(out)


def stream_widths(bits):
    out = []
    for b in range(1, 9):
        out += [b] * (2 * int(np.sum(np.asarray(bits) == b)))
    return np.array(out)


def tol_attention():
    return 2e-3


def sqrt(x):
    return math.sqrt(x)
