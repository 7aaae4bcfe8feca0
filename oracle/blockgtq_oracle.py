"""Plain float64 CPU oracle for the Block-GTQ packed-cache serving path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and imports nothing from it.

Paper: "RoPE-Aware Bit Allocation for KV-Cache Quantization" (Block-GTQ).
Every function names the passage it follows.  Readings taken where the paper
is silent are marked READING and listed in the design notes of the repository.

Conventions (one KV head, head dim d_h, L = d_h / 2 RoPE blocks):
* RoPE block i is the pair of dims (i, i + d_h/2)                 [READING R1]
* bit widths b_i in [1, 8], sum_i b_i = B                          [READING B1]
* codebook: Gaussian Lloyd-Max centroids rounded to fp16, thresholds are the
  midpoints of adjacent fp16 centroids                             [READING Q1]
* a value exactly on a threshold takes the upper code              [READING T2]
* zero vector: stored norm 0, every code 2^(b-1)                   [READING Z1]
* protected window: the first n_sink and last n_recent rows of a context
  use their fp16 K/V, the rest the dequantized ones                 [READING W1]
"""
from __future__ import annotations

import heapq
import math

import numpy as np
from scipy import special

# ---------------------------------------------------------------------------
# Sec. 2.1 (RoPE block notation): R_Delta = diag(R(Delta theta_1), ...), and
# the logit q^T R_Delta k equals the sum of block terms q^(i)T R(Delta theta_i) k^(i).
# ---------------------------------------------------------------------------


def rope_freqs(d_h: int, base: float) -> np.ndarray:
    """theta_i = base^(-2i/d_h), i = 0..L-1                          [READING R1]"""
    return base ** (-2.0 * np.arange(d_h // 2, dtype=np.float64) / d_h)


def block(x: np.ndarray, i: int) -> np.ndarray:
    """The 2-vector x^(i) = (x[i], x[i + d_h/2])."""
    h = x.shape[-1] // 2
    return np.stack([x[..., i], x[..., i + h]], axis=-1)


def rot2(phi: float) -> np.ndarray:
    return np.array([[math.cos(phi), -math.sin(phi)], [math.sin(phi), math.cos(phi)]])


def rope_absolute(x: np.ndarray, pos: float, base: float) -> np.ndarray:
    """R_t x: rotate every block i of x by the angle t * theta_i (Sec. 2.3, R_t)."""
    d = x.shape[-1]
    th = rope_freqs(d, base)
    out = np.empty_like(x, dtype=np.float64)
    h = d // 2
    for i in range(h):
        r = rot2(pos * th[i])
        xi = block(x, i)
        yi = xi @ r.T
        out[..., i] = yi[..., 0]
        out[..., i + h] = yi[..., 1]
    return out


def rope_block_logit(q: np.ndarray, k: np.ndarray, delta: float, base: float) -> float:
    """K_Delta(q, k) = sum_i q^(i)T R(Delta theta_i) k^(i)   (Sec. 2.1)."""
    th = rope_freqs(q.shape[-1], base)
    return float(sum(block(q, i) @ rot2(delta * th[i]) @ block(k, i) for i in range(len(th))))


# ---------------------------------------------------------------------------
# Sec. 3.1, Eq. (scoring-layer-head-energy) and its GQA expansion in the
# calibration appendix: s_i = 1/2 ( mean_{t, g in G(h)} ||q_g,t^(i)||^2
#                                   + mean_t ||k_t^(i)||^2 ).
# ---------------------------------------------------------------------------


def energy_scores(q_cal: np.ndarray, k_cal: np.ndarray) -> np.ndarray:
    """q_cal [N, G, d_h], k_cal [N, d_h] -> s [L] (float64)."""
    q = np.asarray(q_cal, dtype=np.float64)
    k = np.asarray(k_cal, dtype=np.float64)
    n, g, d = q.shape
    h = d // 2
    s = np.empty(h)
    for i in range(h):
        qe = np.sum(q[:, :, i] ** 2 + q[:, :, i + h] ** 2) / (n * g)
        ke = np.sum(k[:, i] ** 2 + k[:, i + h] ** 2) / n
        s[i] = 0.5 * (qe + ke)
    return s


# ---------------------------------------------------------------------------
# Sec. 3.2 objective J(b) = sum_i s_i 4^(-b_i) and Algorithm 1 (greedy
# marginal-gain allocation per layer and KV head).
# ---------------------------------------------------------------------------


def objective(scores, bits) -> float:
    return float(sum(s * 4.0 ** (-b) for s, b in zip(scores, bits)))


def allocate(scores, budget: int, b_min: int = 1, b_max: int = 8) -> np.ndarray:
    """Algorithm 1.  Every block starts at b_min; B_extra = B - L b_min units are
    handed out one at a time to the block with the largest marginal gain
    Delta_i = 3/4 s_i 4^(-b_i).  The constant 3/4 does not change which key is
    largest, so the key used is s_i 4^(-b_i), which is exact in binary floating
    point (a power-of-two scaling).  Equal keys: lowest block index [READING T1].
    """
    s = [float(v) for v in scores]
    L = len(s)
    if budget < L * b_min or budget > L * b_max:
        raise ValueError("infeasible budget")
    b = [b_min] * L
    extra = budget - L * b_min
    heap = [(-math.ldexp(s[i], -2 * b[i]), i) for i in range(L) if b[i] < b_max]
    heapq.heapify(heap)
    while extra > 0 and heap:
        _, i = heapq.heappop(heap)
        b[i] += 1
        extra -= 1
        if b[i] < b_max:
            heapq.heappush(heap, (-math.ldexp(s[i], -2 * b[i]), i))
    return np.array(b, dtype=np.int64)


# ---------------------------------------------------------------------------
# Sec. 2.2 (TQ-MSE local quantizer): normalise, rotate by a shared orthogonal
# matrix, scalar-quantize each rotated coordinate, restore the radius.
# The scalar codebook is not given in the paper; READING Q1: a Gaussian
# Lloyd-Max quantizer for the coordinates of sqrt(d) * (rotated unit vector),
# stored in fp16, with thresholds at the midpoints of adjacent fp16 centroids.
# ---------------------------------------------------------------------------


def _phi(x):
    return np.where(np.isfinite(x), np.exp(-0.5 * np.square(np.where(np.isfinite(x), x, 0.0))) / math.sqrt(2 * math.pi), 0.0)


def _cell_prob(lo, hi):
    """P(lo <= X < hi) for X ~ N(0,1), accurate in both tails."""
    right = lo >= 0
    return np.where(right, special.ndtr(-lo) - special.ndtr(-hi), special.ndtr(hi) - special.ndtr(lo))


def lloyd_max_gaussian(b: int, tol: float = 1e-15, max_iter: int = 200) -> np.ndarray:
    """Centroids of the 2^b-level minimum-MSE scalar quantizer of N(0,1).

    Solves the two Lloyd-Max conditions (each threshold is the midpoint of its
    neighbours, each centroid is the conditional mean of its cell) by Newton's
    method on the fixed-point map c -> E[X | X in cell(c)], started from the
    companded (density^(1/3)) point density.  Returns float64 centroids,
    exactly antisymmetric.
    """
    n = 1 << b
    c = math.sqrt(3.0) * special.ndtri((np.arange(n) + 0.5) / n)
    for _ in range(max_iter):
        t = 0.5 * (c[:-1] + c[1:])
        lo = np.concatenate([[-np.inf], t])
        hi = np.concatenate([t, [np.inf]])
        p = _cell_prob(lo, hi)
        g = (_phi(lo) - _phi(hi)) / p            # conditional means
        # derivatives of g_k w.r.t. its lower / upper threshold
        dlo = np.where(np.isfinite(lo), _phi(lo) * (g - np.where(np.isfinite(lo), lo, 0.0)) / p, 0.0)
        dhi = np.where(np.isfinite(hi), _phi(hi) * (np.where(np.isfinite(hi), hi, 0.0) - g) / p, 0.0)
        jac = np.zeros((n, n))
        for k in range(n):
            if k > 0:      # lower threshold t_{k-1} = (c_{k-1} + c_k)/2
                jac[k, k - 1] += 0.5 * dlo[k]
                jac[k, k] += 0.5 * dlo[k]
            if k < n - 1:  # upper threshold t_k = (c_k + c_{k+1})/2
                jac[k, k] += 0.5 * dhi[k]
                jac[k, k + 1] += 0.5 * dhi[k]
        step = np.linalg.solve(np.eye(n) - jac, g - c)
        c = c + step
        c = 0.5 * (c - c[::-1])
        if np.max(np.abs(step)) < tol:
            break
    return c


def fp16_round(x) -> np.ndarray:
    """Round to the nearest fp16 (ties to even), returned as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


_CB_CACHE: dict = {}


def codebook(b: int):
    """(C16, thresholds): fp16-rounded centroids and the midpoints between
    adjacent fp16 centroids (both float64; the midpoints are exact)."""
    if b not in _CB_CACHE:
        c16 = fp16_round(lloyd_max_gaussian(b))
        _CB_CACHE[b] = (c16, 0.5 * (c16[:-1] + c16[1:]))
    return _CB_CACHE[b]


def scalar_quantize(z: np.ndarray, b: int) -> np.ndarray:
    """code = number of thresholds t with t <= z  (ties go up)    [READING T2]"""
    _, t = codebook(b)
    return np.searchsorted(t, z, side="right").astype(np.int64)


def lloyd_max_mse(b: int, c: np.ndarray | None = None) -> float:
    """E[(X - Q(X))^2] for X ~ N(0,1) with nearest-centroid cells of `c`."""
    if c is None:
        c = lloyd_max_gaussian(b)
    t = 0.5 * (c[:-1] + c[1:])
    lo = np.concatenate([[-np.inf], t])
    hi = np.concatenate([t, [np.inf]])
    # E[(X-c)^2 1{lo<=X<hi}] = m2 - 2 c m1 + c^2 p, with the truncated moments
    p = _cell_prob(lo, hi)
    m1 = _phi(lo) - _phi(hi)
    lo0 = np.where(np.isfinite(lo), lo, 0.0)
    hi0 = np.where(np.isfinite(hi), hi, 0.0)
    m2 = p + lo0 * _phi(lo) - hi0 * _phi(hi)
    return float(np.sum(m2 - 2 * c * m1 + c * c * p))


def tq_encode(x: np.ndarray, rot: np.ndarray, b: int):
    """TQ-MSE encode rows of x [n, d] (Sec. 2.2).

    Returns (codes [n, d] int64, stored norm [n] as fp16-valued float64,
    z [n, d] float64 = the scaled rotated coordinates that were quantized).
    n = ||x||; z = sqrt(d) * Pi x / n; norm stored in fp16 (the radius itself).
    """
    x = np.asarray(x, dtype=np.float64)
    pi = np.asarray(rot, dtype=np.float64)
    d = x.shape[1]
    nrm = np.sqrt(np.sum(x * x, axis=1))
    safe = np.where(nrm > 0, nrm, 1.0)
    z = math.sqrt(d) * (x @ pi.T) / safe[:, None]
    z[nrm == 0] = 0.0                               # READING Z1
    codes = scalar_quantize(z, b)
    return codes, fp16_round(nrm), z


def tq_decode(codes: np.ndarray, norm: np.ndarray, rot: np.ndarray, b: int) -> np.ndarray:
    """x_hat = (norm / sqrt(d)) Pi^T C16[codes]   (rows)."""
    c16, _ = codebook(b)
    pi = np.asarray(rot, dtype=np.float64)
    d = codes.shape[1]
    return (np.asarray(norm, dtype=np.float64)[:, None] / math.sqrt(d)) * (c16[codes] @ pi)


# ---------------------------------------------------------------------------
# Same-rate grouping (end of Sec. 3.2): blocks with equal b form one group
# G_b = {i : b_i = b}; their key blocks are concatenated and encoded by one
# TQ-MSE encoder at b bits/dim.  Order of groups and of dims inside a group
# is not given; READING G1: ascending b, then ascending block index, each
# block contributing (dim i, dim i + d_h/2).
# ---------------------------------------------------------------------------


def groups(bits) -> list:
    """[(b, dims)] for every nonempty same-rate group, ascending b."""
    bits = np.asarray(bits)
    h = len(bits)
    out = []
    for b in range(1, 9):
        members = np.nonzero(bits == b)[0]
        if len(members):
            dims = np.stack([members, members + h], axis=1).reshape(-1)
            out.append((b, dims))
    return out


def quantize_keys(k: np.ndarray, bits, rot_k: dict):
    """Encode key rows k [n, d_h] with the mixed-rate schedule `bits`.

    Returns codes [n, d_h] in stream order (group by group), widths [d_h],
    norms [n, n_groups] (fp16-valued), z [n, d_h] in stream order.
    """
    k = np.asarray(k, dtype=np.float64)
    parts, widths, norms, zs = [], [], [], []
    for b, dims in groups(bits):
        c, nrm, z = tq_encode(k[:, dims], rot_k[len(dims)], b)
        parts.append(c)
        zs.append(z)
        norms.append(nrm)
        widths += [b] * len(dims)
    return (np.concatenate(parts, axis=1), np.array(widths), np.stack(norms, axis=1),
            np.concatenate(zs, axis=1))


def dequantize_keys(codes: np.ndarray, norms: np.ndarray, bits, rot_k: dict) -> np.ndarray:
    """Inverse of quantize_keys: rows in the original dims (post-RoPE coordinates)."""
    n = codes.shape[0]
    out = np.zeros((n, len(bits) * 2))
    col = 0
    for gi, (b, dims) in enumerate(groups(bits)):
        d = len(dims)
        out[:, dims] = tq_decode(codes[:, col:col + d], norms[:, gi], rot_k[d], b)
        col += d
    return out


def quantize_values(v: np.ndarray, rot_v: np.ndarray, b_v: int):
    """V is uniform TQ-MSE over all d_h dims with one norm per token (Sec. 1,
    Sec. 4): returns codes [n, d_h], norms [n], z [n, d_h]."""
    return tq_encode(v, rot_v, b_v)


def dequantize_values(codes, norms, rot_v, b_v):
    return tq_decode(codes, norms, rot_v, b_v)


# ---------------------------------------------------------------------------
# Physical packed layout (READING P1).  The paper stores nibble/byte
# containers; this build packs dense b-bit fields into 32-bit words.
#  K row: codes in stream order, field p at stream bits [o_p, o_p + b_p),
#         o_p = sum of earlier widths; stream bit o is bit (o mod 32) of word
#         floor(o / 32); ceil(sum b / 32) words per row.
#  V tile: 32 tokens; for each rotated coordinate j the 32 codes of the tile
#         form a b_v-word bit string, token slot s at bits [s b_v, s b_v + b_v).
# ---------------------------------------------------------------------------


def pack_key_rows(codes: np.ndarray, widths) -> np.ndarray:
    widths = [int(w) for w in widths]
    n_words = (sum(widths) + 31) // 32
    out = np.zeros((codes.shape[0], n_words), dtype=np.uint64)
    o = 0
    for p, b in enumerate(widths):
        val = codes[:, p].astype(np.uint64) << np.uint64(o % 32)
        out[:, o // 32] |= val & np.uint64(0xFFFFFFFF)
        if o % 32 + b > 32:
            out[:, o // 32 + 1] |= val >> np.uint64(32)
        o += b
    return out.astype(np.uint32)


def unpack_key_rows(words: np.ndarray, widths) -> np.ndarray:
    widths = [int(w) for w in widths]
    w64 = words.astype(np.uint64)
    out = np.zeros((words.shape[0], len(widths)), dtype=np.int64)
    o = 0
    for p, b in enumerate(widths):
        v = w64[:, o // 32] >> np.uint64(o % 32)
        if o % 32 + b > 32:
            v |= w64[:, o // 32 + 1] << np.uint64(32 - o % 32)
        out[:, p] = (v & np.uint64((1 << b) - 1)).astype(np.int64)
        o += b
    return out


def pack_value_tiles(codes: np.ndarray, b_v: int, t0: int = 0, capacity: int | None = None,
                     into: np.ndarray | None = None) -> np.ndarray:
    """Write value codes of tokens t0 .. t0+n-1 into the tile layout
    [capacity/32, d_h, b_v] uint32 (zero-initialised unless `into` is given;
    the bits of other tokens in `into` are kept)."""
    n, d = codes.shape
    if capacity is None:
        capacity = ((t0 + n + 31) // 32) * 32
    out = np.zeros((capacity // 32, d, b_v), dtype=np.uint64) if into is None else into.astype(np.uint64)
    tok = np.arange(t0, t0 + n)
    for s in range(32):                      # token slot inside a tile
        sel = tok % 32 == s
        if not np.any(sel):
            continue
        tiles = tok[sel] // 32
        o = s * b_v
        val = codes[sel].astype(np.uint64) << np.uint64(o % 32)
        field = np.uint64((1 << b_v) - 1) << np.uint64(o % 32)
        out[tiles, :, o // 32] &= ~(field & np.uint64(0xFFFFFFFF))
        out[tiles, :, o // 32] |= val & np.uint64(0xFFFFFFFF)
        if o % 32 + b_v > 32:
            out[tiles, :, o // 32 + 1] &= ~(field >> np.uint64(32))
            out[tiles, :, o // 32 + 1] |= val >> np.uint64(32)
    return out.astype(np.uint32)


def unpack_value_tiles(tiles: np.ndarray, b_v: int, n: int, t0: int = 0) -> np.ndarray:
    w64 = tiles.astype(np.uint64)
    out = np.zeros((n, tiles.shape[1]), dtype=np.int64)
    tok = np.arange(t0, t0 + n)
    for s in range(32):
        sel = tok % 32 == s
        if not np.any(sel):
            continue
        tl = tok[sel] // 32
        o = s * b_v
        v = w64[tl, :, o // 32] >> np.uint64(o % 32)
        if o % 32 + b_v > 32:
            v |= w64[tl, :, o // 32 + 1] << np.uint64(32 - o % 32)
        out[sel] = (v & np.uint64((1 << b_v) - 1)).astype(np.int64)
    return out


# ---------------------------------------------------------------------------
# Decode attention over the packed cache (Sec. 4).  The cache stores
# post-RoPE keys, so the logit of a post-RoPE query is a plain dot product
# with the decoded post-RoPE key (appendix coordinate change); logits carry
# the usual 1/sqrt(d_h) scale, probabilities are a softmax, the output is the
# probability-weighted sum of decoded values.
# ---------------------------------------------------------------------------


def attention(q: np.ndarray, k_hat: np.ndarray, v_hat: np.ndarray) -> np.ndarray:
    """Definition mode.  q [Hg, d], k_hat/v_hat [T, d] -> out [Hg, d]."""
    q = np.asarray(q, dtype=np.float64)
    d = q.shape[-1]
    logits = q @ np.asarray(k_hat, dtype=np.float64).T / math.sqrt(d)
    m = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - m)
    p /= p.sum(axis=1, keepdims=True)
    return p @ np.asarray(v_hat, dtype=np.float64)


def attention_rotated(q, key_codes, key_norms, bits, rot_k, val_codes, val_norms, rot_v, b_v):
    """Algebraically identical rearrangement used as the timed CPU baseline:
    logits = sum_g (n_g / sqrt(d_g)) (Pi_g q_g) . C16[codes_g] / sqrt(d_h) and
    out = Pi_V^T sum_t p_t (n^V_t / sqrt(d_h)) C16[codes^V_t]."""
    q = np.asarray(q, dtype=np.float64)
    d_h = q.shape[-1]
    logits = np.zeros((q.shape[0], key_codes.shape[0]))
    col = 0
    for gi, (b, dims) in enumerate(groups(bits)):
        dg = len(dims)
        c16, _ = codebook(b)
        qg = q[:, dims] @ np.asarray(rot_k[dg], dtype=np.float64).T          # [Hg, dg]
        dots = qg @ c16[key_codes[:, col:col + dg]].T                         # [Hg, T]
        logits += dots * (key_norms[:, gi] / math.sqrt(dg))[None, :]
        col += dg
    logits /= math.sqrt(d_h)
    m = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - m)
    p /= p.sum(axis=1, keepdims=True)
    c16v, _ = codebook(b_v)
    acc = (p * (np.asarray(val_norms) / math.sqrt(d_h))[None, :]) @ c16v[val_codes]
    return acc @ np.asarray(rot_v, dtype=np.float64)


def prefill_attention(q: np.ndarray, q_pos, k_hat: np.ndarray, v_hat: np.ndarray) -> np.ndarray:
    """Causal prefill attention over the cache (Sec. 4, prefill paragraph):
    query row i sits at absolute position q_pos[i] and attends cache rows
    0 .. q_pos[i] (inclusive).  q [n, d], k_hat/v_hat [T, d] with T > max(q_pos)
    -> out [n, d].  Definition mode: one masked softmax per row."""
    q = np.asarray(q, dtype=np.float64)
    pos = np.asarray(q_pos, dtype=np.int64)
    out = np.zeros(q.shape)
    for i in range(q.shape[0]):   # rows past pos are never read
        out[i] = attention(q[i:i + 1], k_hat[:pos[i] + 1], v_hat[:pos[i] + 1])[0]
    return out


def protected_attention(q: np.ndarray, k_hat: np.ndarray, v_hat: np.ndarray, k16: np.ndarray, v16: np.ndarray,
                        n_sink: int, n_recent: int) -> np.ndarray:
    """Decode attention in the protected-buffer regime (Sec. 6, reasoning
    evaluation, and the buffer configurations of its appendix): of a context
    of T rows, the first n_s = min(n_sink, T) and the last
    n_r = min(n_recent, T - n_s) keep their fp16 keys/values (k16, v16,
    [T, d], already fp16-rounded), the rows in between are the dequantized
    ones (k_hat, v_hat).  Definition mode: the keys and values of every row
    are picked, then one softmax over all T rows.  q [Hg, d] -> [Hg, d].
    [READING W1]"""
    T = k_hat.shape[0]
    ns = min(n_sink, T)
    nr = min(n_recent, T - ns)
    fp16_row = np.zeros(T, dtype=bool)
    fp16_row[:ns] = True
    fp16_row[T - nr:] = True
    k = np.where(fp16_row[:, None], np.asarray(k16, dtype=np.float64), np.asarray(k_hat, dtype=np.float64))
    v = np.where(fp16_row[:, None], np.asarray(v16, dtype=np.float64), np.asarray(v_hat, dtype=np.float64))
    return attention(q, k, v)


def attention_partial(q, k_hat, v_hat):
    """(m, l, acc) of one key range: running max, sum of exp, unnormalised output."""
    q = np.asarray(q, dtype=np.float64)
    logits = q @ np.asarray(k_hat, dtype=np.float64).T / math.sqrt(q.shape[-1])
    m = logits.max(axis=1)
    e = np.exp(logits - m[:, None])
    return m, e.sum(axis=1), e @ np.asarray(v_hat, dtype=np.float64)


def lse_merge(parts) -> np.ndarray:
    """Exact log-sum-exp merge of per-range partials (Sec. 4, split-K decode)."""
    m = np.max(np.stack([p[0] for p in parts]), axis=0)
    l = sum(p[1] * np.exp(p[0] - m) for p in parts)
    acc = sum(p[2] * np.exp(p[0] - m)[:, None] for p in parts)
    return acc / l[:, None]
